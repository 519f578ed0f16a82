"""Batches on several streams at once: each call writes only its own buffers,
so two steps running concurrently on two streams (one cache handle, distinct
buffers) give bit for bit what each gives alone."""
import pytest
import torch

from paper_2502_06798_amd import synth
from tests.gpu_check import say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("route,fallback", [("rounds", False), ("planned", True)])
def test_concurrent_steps_equal_sequential(route, fallback):
    import paper_2502_06798_amd as apc
    apc.load()
    say(f"two streams route={route} fallback={fallback}")
    w = synth.BY_NAME["b256_n100k_d768_f16"].scaled(N=40000, latent_shape=(4, 16, 16))
    C = synth.centres(w, "cuda")
    e, es = synth.entries(w, "cuda", C)
    q, qs = synth.queries(w, "cuda", C)
    q2 = q.flip(0).contiguous()                                  # a second batch
    pool = synth.latents(w, "cuda")
    lvl, cap, queue = synth.instances(w)
    theta, K = synth.thresholds(w)
    c = apc.apc_build_cache(e, es, pool, synth.slot_map(w, "cuda"))
    mk = lambda: apc.MatchStep(c, w.B, w.k, theta, K, lvl, cap, queue, latent_bytes=w.latent_bytes,
                               route=route, resident_fallback=fallback)
    a, b = mk(), mk()

    def outs(st):
        return [t.clone() for t in (st.top_score, st.top_idx, st.opt_level, st.out_level, st.out_inst,
                                    st.out_slot, st.inst_fill, st.hit, st.batch)]

    for st in (a, b):
        st.batch.zero_()
    a.run(q, qs)
    torch.cuda.synchronize()
    ref_a = outs(a)
    b.run(q2, qs)
    torch.cuda.synchronize()
    ref_b = outs(b)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for rep in range(6):
        for st in (a, b):
            st.batch.zero_()
        torch.cuda.synchronize()
        a.run(q, qs, stream=s1)
        b.run(q2, qs, stream=s2)
        torch.cuda.synchronize()
        for x, y in zip(ref_a + ref_b, outs(a) + outs(b)):
            assert torch.equal(x, y), f"concurrent run {rep} differs"
    c.close()
