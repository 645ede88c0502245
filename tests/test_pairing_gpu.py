"""Both pairings of row groups inside an attention workgroup (mirrored q with
R-1-q, adjacent 2q with 2q+1), forced through MOCAP_PAIRING, against the
oracle.  The library normally picks one per launch from its time model.
Mirrored pairs whose row groups differ by at least four key tiles share
their last tiles between the two waves of a SIMD (each takes one 32-key
half, the partial results are merged in LDS); the long single chunks below
make most pairs do so."""
import pytest

from helpers import check_chunks, run_gpu, say
from paper_2606_22968_amd import synth

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("mode", ["mirrored", "adjacent"])
@pytest.mark.parametrize("h_q,h_kv,d,lengths,splits", [
    (32, 8, 128, [1536, 768], 0),              # 12 / 6 row groups, automatic split
    (8, 2, 64, [5, 300, 211, 129], 3),         # odd row-group counts, forced split
    (12, 4, 128, [640, 383], 1),               # GQA group 3: one head per unit
    (4, 1, 128, [2048], 0),                    # one causal triangle, 16 mirrored pairs
    (3, 1, 64, [1500, 700], 2),                # one head per unit, head_dim 64, split prefix
])
def test_pairing_matches_oracle(gpu, oracle_lib, monkeypatch, mode, h_q, h_kv, d, lengths, splits):
    monkeypatch.setenv("MOCAP_PAIRING", mode)
    say(f"[case] pairing={mode} h_q={h_q} h_kv={h_kv} d={d} lengths={lengths} splits={splits}")
    q, k, v = synth.make_qkv(400 + d + h_q, sum(lengths), h_q, h_kv, d)
    scale = d ** -0.5
    runner = run_gpu(q, k, v, lengths, scale, block_size=64, num_splits=splits)
    check_chunks(oracle_lib, runner, q, k, v, scale, label=f"pairing {mode}")
