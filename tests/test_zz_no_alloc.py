"""mc_rl_loss_noalloc (the loss entry point that takes no workspace and
allocates nothing; its scratch is a fixed device array inside the library)
against mc_rl_loss, through the C ABI, on two calls in a row: the second
with a smaller batch, so it runs on the scratch the first one left behind.
Both are also held to the oracle's bar."""
import numpy as np
import pytest

import oracle
from _cases import LOSS_RTOL, structure_tensors, to_params
from workloads import make_structure

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_04847_amd as mc
    mc.load_library()


def _outputs(T, B):
    f32 = torch.float32
    return dict(loss=torch.empty(1, dtype=f32, device="cuda"),
                dlogp=torch.full((T,), float("nan"), dtype=f32, device="cuda"),
                seq_mask=torch.empty(B, dtype=torch.uint8, device="cuda"),
                seq_len=torch.empty(B, dtype=torch.int32, device="cuda"),
                n_valid=torch.empty(1, dtype=torch.int64, device="cuda"),
                adv=torch.empty(B, dtype=f32, device="cuda"),
                stat_abs=torch.empty(B, dtype=f32, device="cuda"),
                stat_signed=torch.empty(B, dtype=f32, device="cuda"),
                clip_frac=torch.empty(1, dtype=f32, device="cuda"),
                error_flag=torch.empty(1, dtype=torch.int32, device="cuda"),
                kl=torch.empty(1, dtype=f32, device="cuda"),
                token_frac=torch.empty(1, dtype=f32, device="cuda"))


def _case(cid, seed, p):
    import paper_2606_04847_amd as mc
    s = make_structure(cid)
    rng = np.random.default_rng(seed)
    logp = (-rng.uniform(0.5, 12.0, size=s.T)).astype(np.float32)
    lr = (logp.astype(np.float64) + s.rollout_delta).astype(np.float32)
    st = structure_tensors(s)
    lp, lrd = torch.from_numpy(logp).cuda(), torch.from_numpy(lr).cuda()
    args = (lp, lrd, st["mask"], st["cu"], st["cg"], st["rewards"], to_params(p))
    ref = mc.rl_loss(*args)                                   # workspace entry point
    out = _outputs(s.T, s.B)
    got = mc.rl_loss(*args, out=out, noalloc=True)            # no workspace, no allocation
    torch.cuda.synchronize()
    o = oracle.rl_loss(logp, lr, s.loss_mask, s.cu_seqlens, s.cu_groups, s.rewards, p)
    return ({k: v.cpu().numpy() for k, v in ref.items()},
            {k: v.cpu().numpy() for k, v in got.items()}, o)


def _check(ref, got, o):
    for k in ref:
        assert np.array_equal(ref[k], got[k], equal_nan=True), k   # same kernels, same order
    assert got["error_flag"][0] == 0
    assert np.array_equal(got["seq_mask"], o["seq_mask"])
    assert np.array_equal(got["seq_len"], o["seq_len"])
    assert int(got["n_valid"][0]) == o["n_valid"]
    assert abs(got["loss"][0] - o["loss"]) <= LOSS_RTOL * max(abs(o["loss"]), 1e-30)
    np.testing.assert_allclose(got["dlogp"], o["dlogp"], rtol=1e-5, atol=1e-12)


def test_noalloc_loss_matches_the_workspace_entry_point_twice():
    # first call: the 256-sequence filter-stress batch with IcePop; second:
    # the 16-sequence batch (fewer sequences and groups) on the same scratch
    p1 = oracle.RLParams(token_mode="icepop", icepop_lo=0.75, icepop_hi=1.3)
    _check(*_case(4, 300, p1))
    _check(*_case(1, 301, oracle.RLParams()))


def test_noalloc_loss_rejects_batches_beyond_its_scratch():
    import ctypes
    import paper_2606_04847_amd as mc
    from paper_2606_04847_amd import binding
    lib = mc.load_library()
    cap = lib.mc_rl_loss_noalloc_max_bytes()
    B = 1 << 20                                  # far beyond 4 MiB of per-sequence scratch
    assert lib.mc_rl_loss_workspace_size(B, B, 1) > cap
    dummy = torch.zeros(16, device="cuda")
    o = binding.RLOutputsC(dummy.data_ptr(), dummy.data_ptr(),
                           *([None] * (len(binding._OUT_FIELDS) - 2)))
    pc = binding.RLParams().to_c()
    st = lib.mc_rl_loss_noalloc(dummy.data_ptr(), dummy.data_ptr(), None, None,
                                dummy.data_ptr(), dummy.data_ptr(), dummy.data_ptr(), B, B, 1,
                                ctypes.byref(pc), ctypes.byref(o), None)
    assert st == binding.MC_ERR_UNSUPPORTED
