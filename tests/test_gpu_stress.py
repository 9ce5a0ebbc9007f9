"""GPU: the graph-replay stress run (preset 5; Alg. 2 and Eq. (13)).

36 layers of Qwen3-8B-shaped verify attention (32q/8kv, D=128, 36 distinct
KV pools) plus acceptance over a 151,936-token vocabulary, B=32, for 100
consecutive steps.  Each step redraws the verify lengths and drafts,
regenerates the planted logits, and grows every context by its accepted
count plus one; all metadata lives in fixed-address buffers and one hipGraph
captured before the first step is replayed every step.  Checked: the
acceptance of every step against the planted values (exact), and the
attention rows of sampled (step, layer, request) triples against the fp64
oracle (max-abs 1e-2, mean-abs 1e-3).
"""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

try:
    from gpu_util import say
    from workloads.stress import StressRun
except Exception:  # pragma: no cover
    pass

SAMPLED_STEPS = (0, 37, 99)


def check_attention(run, st, layer, step):
    live = [i for i in range(run.plan.B) if st.qlens[i] > 0]
    reqs = sorted({live[0], live[-1], max(live, key=lambda i: st.qlens[i])})
    g = run.gather_request_inputs(layer, reqs, st)
    ref = oracle.verify_attn(g["q"], g["cu_qlens"], g["kv_pages"], g["page_table"],
                             g["ctx_lens"], num_q_heads=run.hq, num_kv_heads=run.hkv,
                             head_dim=run.d, page_size=16, scale=1.0 / np.sqrt(run.d))
    got = W.bf16_to_f32(g["out_bits"]).astype(np.float64)
    err = np.abs(got - ref)
    say("stress", "step %d layer %d requests %s: max %.3g mean %.3g"
        % (step, layer, reqs, err.max(), err.mean()))
    assert np.isfinite(got).all()
    assert err.max() <= 1e-2 and err.mean() <= 1e-3


def test_graph_replay_stress_36_layers_100_steps():
    plan = W.StressPlan()
    say("stress", "layers %d, B %d, steps %d, pool %d pages per layer, max_kv_len %d"
        % (plan.num_layers, plan.B, plan.steps, plan.num_pages, plan.max_kv_len))
    run = StressRun(plan)
    first = plan.draw_step()
    run.stage(first)
    run.capture()
    addrs = (run.cu.data_ptr(), run.ctx.data_ptr(), run.logits.data_ptr())
    ctx_start = run.ctx_host.copy()
    st = first
    for step in range(plan.steps):
        if step > 0:
            st = plan.draw_step()
            run.stage(st)
        run.replay()
        a, nxt = run.finish(st)
        assert (a == st.planted_accept_len).all(), (step, a, st.planted_accept_len)
        assert (nxt == st.planted_next).all(), step
        if step in SAMPLED_STEPS:
            for layer in (0, plan.num_layers - 1):
                check_attention(run, st, layer, step)
    # the buffers never moved, and the contexts grew by accepted + 1 per step
    assert addrs == (run.cu.data_ptr(), run.ctx.data_ptr(), run.logits.data_ptr())
    grown = run.ctx_host - ctx_start
    say("stress", "contexts grew by %d..%d tokens over %d steps" % (grown.min(), grown.max(),
                                                                    plan.steps))
    assert (grown >= plan.steps).all()
    run.close()
