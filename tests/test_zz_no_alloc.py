"""The allocation-free planner entry point, buddy_pool_route_noalloc,
through the C ABI against buddy_pool_route on the same inputs.

Both run the same kernels with the same pool split count, so the scores
must agree bit for bit.  Each case makes two calls in a row on the
device's shared scratch array, the second with a smaller input (fewer
sequences, shorter contexts, one shared position instead of per-sequence
ones), so stale scratch contents from the first call cannot leak into the
second.  A batch whose buffers exceed the scratch array is refused with
BUDDY_ECAPACITY and nothing written.
"""
import pytest
import torch

from paper_2606_09514_amd import lib as blib
from paper_2606_09514_amd import synth

from _gpu import Pair

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("running", [False, True], ids=["scan", "running_sums"])
@pytest.mark.parametrize("dtype,shape", [("f32", "tiny"), ("bf16", "tiny"), ("bf16", "llama3_8b")])
def test_pool_route_noalloc_matches_pool_route(dtype, shape, running):
    Bcap, T = 6, 300
    P = Pair(shape, dtype, T, Bcap, seed=3, omega=0.1, device_gen=(shape != "tiny"))
    g = torch.Generator().manual_seed(9)
    dk = P.upload(synth.storage_numpy(torch.randn(P.shape5, generator=g).to(P.tdt)))
    dv = P.upload(synth.storage_numpy(torch.randn(P.shape5, generator=g).to(P.tdt)))
    h = synth.hidden_inputs(Bcap, P.cfg["d_model"], seed=10).cuda()
    for pos in ([T - 1, 0, 17, 63, 150, 298], [5, 5, 5]):
        B = len(pos)
        hb = h[:B].contiguous()
        ref = torch.full((B, P.L_mid), float("nan"), device="cuda")
        got = torch.full((B, P.L_mid), float("nan"), device="cuda")
        # running sums: both calls start from the same (zeroed) state
        pool_a = P.gpu.pool_state() if running else None
        pool_b = P.gpu.pool_state() if running else None
        P.gpu.pool_route(dk, dv, pos, hb, ref, pool=pool_a)
        blib.pool_route_noalloc(P.cfg, P.Wd["dm"], Bcap, dk, dv, pos, hb, got, pool=pool_b)
        torch.cuda.synchronize()
        assert torch.equal(got.cpu(), ref.cpu()), (pos, (got - ref).abs().max().item())
        assert torch.isfinite(got).all()
        if running:
            assert torch.equal(pool_a[0].cpu(), pool_b[0].cpu())
            assert torch.equal(pool_a[1].cpu(), pool_b[1].cpu())


def test_pool_route_noalloc_refuses_batches_beyond_the_scratch():
    """A 40-KV-head shape at B = 200 needs more than the 8 MiB scratch (its
    pool partials, 200 x 40 x 1 KB, and the Decision Module's activations
    come to 8.6 MB): BUDDY_ECAPACITY before anything is enqueued."""
    cfg = synth.model_config("mha_13b", "bf16", 64)
    small = lambda *s, dt=torch.bfloat16: torch.zeros(s, dtype=dt, device="cuda")
    dm = dict(w1=small(8), b1=small(8), w2=small(8), b2=small(8), prior=None, omega=0.0)
    kc, vc = small(8), small(8)
    h = small(200, cfg["d_model"], dt=torch.float32)
    out = torch.full((200, cfg["n_layers"] - 2), 7.0, device="cuda")
    rc = blib.pool_route_noalloc(cfg, dm, 256, kc, vc, [10] * 200, h, out, check=False)
    torch.cuda.synchronize()
    assert rc == 3                                   # BUDDY_ECAPACITY
    assert torch.all(out == 7.0)
    # a batch above the cache capacity is refused as well
    rc = blib.pool_route_noalloc(cfg, dm, 150, kc, vc, [10] * 160, h[:160].contiguous(),
                                 out[:160].contiguous(), check=False)
    assert rc == 3
