"""A whole matching step captured as a HIP graph: every replay, with eager
work and synchronisations in between, equals the eager step bit for bit."""
import pytest
import torch

from paper_2502_06798_amd import synth
from tests.gpu_check import say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,B,N,route,fallback", [("b256_n100k_d768_f16", 256, 20000, "rounds", False),
                                                     ("b16_n10k_d768_f32", 16, 3000, "rounds", False),
                                                     ("b256_n100k_d768_f16", 256, 20000, "planned", True),
                                                     ("b1024_n1m_d768_bf16", 1024, 30000, "planned", True)])
def test_step_graph_replays_equal_eager(name, B, N, route, fallback):
    import paper_2502_06798_amd as apc
    apc.load()
    say(f"graph {name} B={B} N={N} route={route} fallback={fallback}")
    w = synth.BY_NAME[name].scaled(B=B, N=N, latent_shape=(4, 16, 16))
    C = synth.centres(w, "cuda")
    e, es = synth.entries(w, "cuda", C)
    q, qs = synth.queries(w, "cuda", C)
    pool = synth.latents(w, "cuda")
    soe = synth.slot_map(w, "cuda")
    lvl, cap, queue = synth.instances(w)
    theta, K = synth.thresholds(w)
    c = apc.apc_build_cache(e, es, pool, soe)
    step = apc.MatchStep(c, w.B, w.k, theta, K, lvl, cap, queue, latent_bytes=w.latent_bytes, route=route,
                         resident_fallback=fallback)
    extra = [t for t in (step.plan, step.res_score, step.res_idx) if t is not None]

    def outputs():
        return [t.clone() for t in [step.top_score, step.top_idx, step.opt_level, step.out_level, step.out_inst,
                                    step.out_slot, step.inst_fill, step.hit, step.batch] + extra]

    def scribble():
        # every output overwritten; latent slots the step leaves empty keep it
        for t in [step.top_score, step.top_idx, step.out_level, step.out_inst, step.out_slot, step.hit] + extra:
            t.fill_(-7)
        step.batch.fill_(3)

    scribble()
    step.run(q, qs)
    torch.cuda.synchronize()
    ref = outputs()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step.run(q, qs)
    for rep in range(4):
        scribble()                                   # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(ref, outputs()):
            assert torch.equal(a, b) or (a.is_floating_point() and torch.equal(a.nan_to_num(9.0), b.nan_to_num(9.0))), \
                f"replay {rep} differs from the eager step"
    del g
    c.close()
