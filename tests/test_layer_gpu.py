"""The per-chunk decoder layer used to measure both terms of Eq. (1): its
attention is exactly the library's chunked attention on the projected
queries/keys/values, and the whole layer output is finite."""
import pytest
import torch

from helpers import check_chunks, say
from paper_2606_22968_amd import lbcp
from paper_2606_22968_amd.layer import ChunkedLayer, LayerShape
from paper_2606_22968_amd.prefill import ChunkedPrefill

pytestmark = pytest.mark.gpu


def test_layer_attention_is_library_attention(gpu, oracle_lib):
    shape = LayerShape("small", 512, 8, 2, 64, 1024)
    lengths = [256, 100, 300, 68]
    S = sum(lengths)
    say(f"[case] layer {shape} lengths={lengths}")
    g = torch.Generator(device="cpu")
    g.manual_seed(5)
    x = torch.randn((S, shape.hidden), generator=g, dtype=torch.float32).to(torch.bfloat16).cuda()
    layer = ChunkedLayer(shape, lengths, seed=6, block_size=64)
    scale = shape.head_dim ** -0.5
    out = layer.run(x, scale)
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all()
    q, k, v = layer.project_qkv(x)
    ref = ChunkedPrefill(shape.h_q, shape.h_kv, shape.head_dim, lengths, block_size=64)
    ref.run(q, k, v, scale)
    torch.cuda.synchronize()
    assert torch.equal(layer.attn.o.view(torch.int16), ref.o.view(torch.int16))
    check_chunks(oracle_lib, ref, q.cpu(), k.cpu(), v.cpu(), scale, label="layer attention")


def test_layer_latency_split(gpu):
    shape = LayerShape("small", 1024, 16, 4, 128, 2048)
    plans = [[1024, 1024, 1024, 1024]]
    rows = lbcp.measure_layer(shape, plans, reps=2, seed=3)
    say(f"[layer] {rows}")
    assert len(rows) == 4
    for _, c, p, total, attn, gemm in rows:
        assert total > 0 and attn > 0 and gemm > 0 and abs(total - attn - gemm) < 1e-6
    # Attention grows with the prefix; the projections do not.
    assert rows[-1][4] > rows[0][4]
