"""The per-chunk decoder layer used to measure both terms of Eq. (1): its
attention is exactly the library's chunked attention on the projected
queries/keys/values, and the whole layer output matches the same layer
computed in fp32 on the CPU from the same weights."""
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


def _cpu_layer(shape, x, w_qkv, w_o, w_gu, w_d, dtype):
    """The decoder layer of layer.py over the whole sequence (chunking does
    not change the result): GEMMs, monolithic causal attention (bottom-right
    aligned, GQA heads repeated), residuals and SwiGLU, every GEMM output
    rounded to `dtype`; attention itself in fp32."""
    S, d = x.shape[0], shape.head_dim
    x = x.to(dtype)
    qkv = x @ w_qkv.to(dtype)
    nq, nk = shape.h_q * d, shape.h_kv * d
    q = qkv[:, :nq].reshape(S, shape.h_q, d).float()
    k = qkv[:, nq:nq + nk].reshape(S, shape.h_kv, d).float().repeat_interleave(shape.h_q // shape.h_kv, 1)
    v = qkv[:, nq + nk:].reshape(S, shape.h_kv, d).float().repeat_interleave(shape.h_q // shape.h_kv, 1)
    s = torch.bmm(q.transpose(0, 1), k.permute(1, 2, 0).contiguous()) * d ** -0.5
    s.masked_fill_(torch.triu(torch.ones(S, S, dtype=torch.bool), 1), float("-inf"))
    o = torch.bmm(torch.softmax(s, -1), v.transpose(0, 1).contiguous()).transpose(0, 1)
    y = x + o.to(dtype).reshape(S, -1) @ w_o.to(dtype)
    gu = y @ w_gu.to(dtype)
    h = torch.nn.functional.silu(gu[:, :shape.ffn]) * gu[:, shape.ffn:]
    return (y + h @ w_d.to(dtype)).float()


def test_layer_output_matches_fp32_cpu_layer(gpu):
    # The GPU layer rounds every GEMM output to bf16 (and attention's
    # probabilities and output, as the library does).  The bar is twice the
    # error that the same bf16 rounding points give when torch computes the
    # layer on the CPU, against the fp32 CPU layer.
    shape = LayerShape("small", 512, 8, 2, 64, 1024)
    lengths = [256, 100, 300, 68]
    S = sum(lengths)
    g = torch.Generator(device="cpu")
    g.manual_seed(5)
    x = torch.randn((S, shape.hidden), generator=g, dtype=torch.float32).to(torch.bfloat16)
    layer = ChunkedLayer(shape, lengths, seed=6, block_size=64)
    out = layer.run(x.cuda(), shape.head_dim ** -0.5).float().cpu()
    w = [t.cpu() for t in (layer.w_qkv, layer.w_o, layer.w_gu, layer.w_d)]
    ref = _cpu_layer(shape, x, *w, torch.float32)
    emu = _cpu_layer(shape, x, *w, torch.bfloat16)
    e_gpu, e_emu = (out - ref).abs(), (emu - ref).abs()
    rel_gpu = ((out - ref).norm() / ref.norm()).item()
    rel_emu = ((emu - ref).norm() / ref.norm()).item()
    say(f"[layer] vs fp32: GPU max {e_gpu.max().item():.3e} mean {e_gpu.mean().item():.3e} rel {rel_gpu:.3e}; "
        f"CPU bf16 max {e_emu.max().item():.3e} mean {e_emu.mean().item():.3e} rel {rel_emu:.3e}")
    assert torch.isfinite(out).all()
    assert e_gpu.max().item() <= 2 * e_emu.max().item()
    assert e_gpu.mean().item() <= 2 * e_emu.mean().item()
    assert rel_gpu <= 2 * rel_emu
