"""A chunk behind a prefix of about a million tokens (8B heads): positions,
block indices and byte offsets far beyond what the other workloads reach
(the K pool alone spans more than 2 GiB), checked against the oracle on
sampled rows, unsplit and with the automatic split plan."""
import numpy as np
import pytest
import torch

from helpers import LSE_MAX_ABS, O_MAX_ABS, O_MEAN_ABS, errors, say
from paper_2606_22968_amd import binding, synth

pytestmark = pytest.mark.gpu

P = (1 << 20) + 64
L = 300
H_Q, H_KV, D = 32, 8, 128
BS = 256


def test_million_token_prefix(gpu, oracle_lib):
    scale = D ** -0.5
    say(f"[case] P={P} L={L}: generating inputs")
    k, v = synth.make_kv_long(91, P + L, H_KV, D)
    q = synth.make_qkv(92, L, H_Q, H_KV, D)[0]
    n_blocks = (P + L + BS - 1) // BS
    table = synth.permuted_table(n_blocks, 93, n_blocks + 64).cuda()
    store = binding.KvStore(n_blocks + 64, BS, H_KV, D, fill=float("nan"))
    say("[case] appending the prefix and the chunk")
    piece = 1 << 16
    for start in range(0, P + L, piece):
        end = min(start + piece, P + L)
        binding.mocap_kv_append(store, table, start, k[start:end].cuda(), v[start:end].cuda())
    torch.cuda.synchronize()
    qd = q.cuda()
    rows = synth.sample_rows(L, 94, n_random=3)
    ref_o, ref_lse = oracle_lib.chunk_attn(synth.bf16_bits(q), synth.bf16_bits(k), synth.bf16_bits(v), P, scale,
                                           rows=rows)
    for splits in (1, 0):
        r, ws_bytes = binding.mocap_chunk_attn_workspace_size(P, L, H_Q, H_KV, D, splits)
        ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device="cuda")
        o = torch.full((L, H_Q, D), float("nan"), dtype=torch.bfloat16, device="cuda")
        lse = torch.full((H_Q, L), float("nan"), dtype=torch.float32, device="cuda")
        binding.mocap_chunk_attn(store, table, qd, P, scale, o, lse, ws, splits)
        torch.cuda.synchronize()
        mx, mean, lmx = errors(o.cpu()[rows], lse.cpu()[:, rows], ref_o, ref_lse)
        say(f"[parity] P={P} splits={splits} ranges={r}: O max-abs {mx:.3e} mean-abs {mean:.3e} LSE {lmx:.3e}")
        assert np.isfinite(mx) and np.isfinite(lmx)
        assert mx <= O_MAX_ABS and mean <= O_MEAN_ABS and lmx <= LSE_MAX_ABS
        assert torch.isfinite(o.float()).all() and torch.isfinite(lse).all()
