"""LBCP stage 1 on the GPU: measured per-chunk latency, the fitted model of
Eq. (1), the dynamic program's plan (Section 4.2, Alg. 1), and parity of the
attention under that plan."""
import pytest

from helpers import check_chunks, run_gpu, say, workload_inputs
from paper_2606_22968_amd import lbcp, synth

pytestmark = pytest.mark.gpu


def test_measured_model_plan_and_parity(gpu, oracle_lib):
    h_q, h_kv, d, S, M, align = 32, 8, 128, 16384, 8, 128
    scale = 1.0 / d ** 0.5
    probes = lbcp.probe_plans(S, M, align, seed=11, n_random=2)
    say(f"[lbcp] measuring {len(probes)} plans of S={S} M={M}")
    samples = lbcp.measure(h_q, h_kv, d, probes, scale, reps=2, seed=11)
    assert len(samples) == len(probes) * M and all(t > 0 for *_, t in samples)
    model = lbcp.fit([(c, p, t) for _, c, p, t in samples])
    say(f"[lbcp] model {model}")
    assert model.cost_pair > 0 and model.rms_rel_err < 0.5
    lengths, t_max, t_sum = lbcp.plan(S, M, 8, align, model)
    assert sum(lengths) == S and all(c % align == 0 and c > 0 for c in lengths)
    # Under the model, the plan's largest chunk cost is no worse than that of
    # the uniform or the closed-form balanced plan.
    for other in probes[:2]:
        costs, p = [], 0
        for c in other:
            costs.append(model(c, p))
            p += c
        assert t_max <= max(costs) * (1 + 1e-9)
    q, k, v = workload_inputs(11, S, h_q, h_kv, d)
    runner = run_gpu(q, k, v, lengths, scale)
    check_chunks(oracle_lib, runner, q, k, v, scale,
                 rows_of=lambda c, n: synth.sample_rows(n, 500 + c, n_random=11),
                 label=f"lbcp plan {lengths}")
