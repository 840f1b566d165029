"""The C ABI: libmc.so loads without a GPU, exports every function that
include/mc.h declares, and rejects bad arguments on the host before any
launch (these calls make no HIP call, so they run here without a GPU)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_04847_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mc.h")

OK, INVALID, UNSUP, WS = 0, 1, 2, 3
F32, BF16 = 0, 1
FAKE = 1 << 20          # an aligned, never-dereferenced address
FAKE_WS = 1 << 24       # 256-byte aligned


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("libmc.so not built")
    return binding.load_library()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]*?\b(mc_\w+)\s*\(", text, re.M)))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert {"mc_logprob_fwd", "mc_logprob_bwd", "mc_rl_loss", "mc_check_packing",
            "mc_status_string", "mc_version"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings_and_version(lib):
    assert binding.status_string(0) == "MC_OK"
    assert binding.status_string(3) == "MC_ERR_WORKSPACE"
    assert "gfx950" in binding.version()


def fwd(lib, T=16, d=64, V=100, dt=BF16, H=FAKE, W=FAKE, y=FAKE, lp=FAKE, ls=FAKE,
        ws=FAKE_WS, nbytes=None):
    need = lib.mc_logprob_fwd_workspace_size(max(T, 0), d, V, dt)
    return lib.mc_logprob_fwd(H, W, y, T, d, V, dt, lp, ls, None, ws,
                              need if nbytes is None else nbytes, None)


def test_fwd_argument_checks(lib):
    assert fwd(lib, T=-1) == INVALID
    assert fwd(lib, d=0) == INVALID
    assert fwd(lib, V=0) == INVALID
    assert fwd(lib, d=60) == UNSUP
    assert fwd(lib, dt=7) == UNSUP
    assert fwd(lib, H=None) == INVALID
    assert fwd(lib, y=None) == INVALID
    assert fwd(lib, ls=None) == INVALID
    assert fwd(lib, H=FAKE + 8) == INVALID          # hidden not 16-byte aligned
    assert fwd(lib, nbytes=10) == WS
    assert fwd(lib, ws=None) == WS
    assert fwd(lib, ws=FAKE_WS + 128) == WS        # workspace not 256-byte aligned
    assert fwd(lib, T=0, H=None, W=None, y=None, lp=None, ls=None, ws=None) == OK  # no-op
    assert fwd(lib, V=1 << 31) == UNSUP


def test_workspace_sizes(lib):
    a = lib.mc_logprob_fwd_workspace_size(1000, 128, 1000, BF16)
    b = lib.mc_logprob_fwd_workspace_size(2000, 128, 1000, BF16)
    assert 0 < a < b
    assert lib.mc_logprob_fwd_workspace_size(10, 60, 10, BF16) == 0      # invalid -> 0
    bw = lib.mc_logprob_bwd_workspace_size(16384, 4096, 151936, BF16)
    # the headline shape keeps its whole 2-byte softmax operand (one chunk),
    # the transposes of W and H, a copy of H with the dead tokens' rows
    # zeroed (in the live-first token order), small index arrays, the fp32
    # slots of dW's split last round (at most 256 tiles of 256 x 256) and the
    # one-hot scatter's two fp32 rows per segment of 16 bucketed tokens
    def seg(T, d):
        return 2 * (-(-T // 16)) * d * 4
    dense = (151936 * 16384 + 4096 * 151936 + 2 * 4096 * 16384) * 2
    assert dense + seg(16384, 4096) <= bw < dense + seg(16384, 4096) + (16 << 20) + (64 << 20)
    # larger problems are chunked under 8 GiB of softmax operand per chunk;
    # the W transpose covers one chunk
    big = lib.mc_logprob_bwd_workspace_size(65536, 4096, 248320, BF16)
    chunk = (8 << 30) // (65536 * 2)
    assert big <= ((8 << 30) + (4096 * chunk + 2 * 4096 * 65536) * 2 + seg(65536, 4096)
                   + (32 << 20) + (64 << 20))
    assert lib.mc_rl_loss_workspace_size(100, 8, 2) > 0
    assert lib.mc_rl_loss_workspace_size(-1, 8, 2) == 0


def bwd(lib, T=16, d=64, V=100, dt=BF16, dh=FAKE, dw=FAKE, flags=0, lse=FAKE, dl=FAKE,
        nbytes=None):
    need = lib.mc_logprob_bwd_workspace_size(T, d, V, dt)
    return lib.mc_logprob_bwd(FAKE, FAKE, FAKE, lse, dl, T, d, V, dt, dh, dw, flags, FAKE_WS,
                              need if nbytes is None else nbytes, None)


def test_bwd_argument_checks(lib):
    assert bwd(lib, dh=None, dw=None) == INVALID
    assert bwd(lib, flags=8) == INVALID            # unknown flag bit
    assert bwd(lib, flags=4, lse=None) == INVALID  # MC_BWD_SKIP_DEAD_TOKENS is known; null lse
    assert bwd(lib, d=12) == UNSUP
    assert bwd(lib, lse=None) == INVALID
    assert bwd(lib, dl=None) == INVALID
    assert bwd(lib, dh=FAKE + 4) == INVALID
    assert bwd(lib, nbytes=0) == WS


def loss(lib, T=10, B=2, NG=1, params=None, out=None, ws=FAKE_WS, nbytes=None, **ptrs):
    p = params or binding.RLParams().to_c()
    o = out or binding.RLOutputsC(FAKE, FAKE, *([None] * (len(binding._OUT_FIELDS) - 2)))
    need = lib.mc_rl_loss_workspace_size(T, B, NG)
    args = dict(logp=FAKE, lr=FAKE, mask=None, cu=FAKE, cg=FAKE, rw=FAKE)
    args.update(ptrs)
    return lib.mc_rl_loss(args["logp"], args["lr"], None, args["mask"], args["cu"], args["cg"],
                          args["rw"], T, B, NG, ctypes.byref(p), ctypes.byref(o), ws,
                          need if nbytes is None else nbytes, None)


@pytest.mark.parametrize("field,value", [
    ("eps_low", 1.0), ("eps_low", -0.1), ("eps_high", -0.5), ("delta", -1.0),
    ("delta", float("nan")), ("adv_eps", float("inf")), ("std_ddof", 2), ("filter", 3),
    ("kl_beta", -0.1), ("kl_beta", float("nan")), ("token_mode", 3), ("token_mode", -1),
])
def test_loss_parameter_checks(lib, field, value):
    p = binding.RLParams().to_c()
    setattr(p, field, value)
    assert loss(lib, params=p) == INVALID


@pytest.mark.parametrize("mode,field,value,ok", [
    ("tis", "tis_cap", 0.0, False), ("tis", "tis_cap", -1.0, False),
    ("tis", "tis_cap", float("inf"), False), ("tis", "tis_cap", 0.5, True),
    ("icepop", "icepop_lo", 0.0, False), ("icepop", "icepop_hi", 0.4, False),
    ("icepop", "icepop_hi", float("nan"), False), ("icepop", "icepop_lo", 1.0, True),
    ("none", "tis_cap", -1.0, True),          # parameters of an unused mode are not read
])
def test_token_mode_parameter_checks(lib, mode, field, value, ok):
    # a valid parameter set passes the parameter checks and stops at the
    # (deliberately short) workspace check, before any launch
    p = binding.RLParams(token_mode=mode).to_c()
    setattr(p, field, value)
    assert loss(lib, params=p, nbytes=1) == (WS if ok else INVALID)


def test_loss_argument_checks(lib):
    assert loss(lib, T=-1) == INVALID
    assert loss(lib, B=0, NG=0) == INVALID            # tokens but no sequence
    assert loss(lib, NG=0) == INVALID                 # sequences but no group
    assert loss(lib, logp=None) == INVALID
    assert loss(lib, cu=None) == INVALID
    assert loss(lib, rw=None) == INVALID
    o = binding.RLOutputsC(None, FAKE, *([None] * (len(binding._OUT_FIELDS) - 2)))
    assert loss(lib, out=o) == INVALID                # loss output is required
    o = binding.RLOutputsC(FAKE, None, *([None] * (len(binding._OUT_FIELDS) - 2)))
    assert loss(lib, out=o) == INVALID                # dlogp output is required
    assert loss(lib, nbytes=1) == WS


def test_host_packing_check(lib):
    good_cu, good_cg = np.array([0, 3, 3, 7]), np.array([0, 1, 3])
    assert binding.check_packing(good_cu, good_cg, 7)
    assert not binding.check_packing(good_cu, good_cg, 8)                # end != T
    assert not binding.check_packing(np.array([1, 3, 3, 7]), good_cg, 7)  # start != 0
    assert not binding.check_packing(np.array([0, 4, 3, 7]), good_cg, 7)  # decreasing
    assert not binding.check_packing(good_cu, np.array([0, 1, 2]), 7)    # groups end != B
    assert not binding.check_packing(good_cu, np.array([0, 2, 1, 3]), 7)
    assert binding.check_packing(np.array([0]), np.array([0]), 0)         # empty batch


def test_shard_and_primeecho_argument_checks(lib):
    need = lib.mc_logprob_fwd_workspace_size(16, 64, 100, BF16)
    call = lambda vs, off, vt: lib.mc_logprob_fwd_shard(FAKE, FAKE, FAKE, 16, 64, vs, off, vt,
                                                        BF16, FAKE, FAKE_WS, need, None)
    assert call(100, -1, 300) == INVALID        # negative offset
    assert call(100, 250, 300) == INVALID       # shard past the vocabulary
    assert call(100, 0, 50) == INVALID          # vocabulary smaller than the shard
    assert lib.mc_logprob_merge_shards(FAKE, 0, FAKE, 16, 100, FAKE, FAKE, None, None) == INVALID
    assert lib.mc_logprob_merge_shards(None, 2, FAKE, 16, 100, FAKE, FAKE, None, None) == INVALID
    bneed = lib.mc_logprob_bwd_workspace_size(16, 64, 100, BF16)
    assert lib.mc_logprob_bwd_shard(FAKE, FAKE, FAKE, FAKE, FAKE, 16, 64, 100, 201, 300, BF16,
                                    FAKE, FAKE, 0, FAKE_WS, bneed, None) == INVALID
    pe = lambda B, K, a, b1: lib.mc_primeecho_rewards(FAKE, None, None, B, K, a, b1, 0.0, FAKE,
                                                      None)
    assert pe(4, 0, 0.75, 0.0) == INVALID       # Kmax < 1
    assert pe(-1, 3, 0.75, 0.0) == INVALID
    assert pe(4, 3, 1.5, 0.0) == INVALID        # alpha outside [0, 1]
    assert pe(4, 3, 0.5, float("inf")) == INVALID
    assert pe(0, 3, 0.5, 0.0) == OK             # no trajectories: no-op


def test_cached_argument_checks(lib):
    T, d, V = 16, 64, 100
    need_c = lib.mc_logprob_cache_size(T, d, V, BF16)
    need_f = lib.mc_logprob_fwd_workspace_size(T, d, V, BF16)
    need_b = lib.mc_logprob_bwd_cached_workspace_size(T, d, V, BF16)
    # the cache holds the padded [T x V] exp operand and the block maxima
    assert need_c >= 64 * 128 * 2 + 16 * 4 and lib.mc_logprob_cache_size(T, 60, V, BF16) == 0
    # the cached backward's workspace holds the gathered operand like the
    # recompute backward's (one chunk here)
    assert 0 < need_b <= lib.mc_logprob_bwd_workspace_size(T, d, V, BF16)
    fwd = lambda cache, cb, ws=FAKE_WS, wb=need_f: lib.mc_logprob_fwd_cached(
        FAKE, FAKE, FAKE, T, d, V, BF16, FAKE, FAKE, None, cache, cb, ws, wb, None)
    assert fwd(None, need_c) == WS
    assert fwd(FAKE_WS, need_c - 1) == WS
    assert fwd(FAKE_WS + 128, need_c) == WS        # cache not 256-byte aligned
    assert fwd(FAKE_WS, need_c, wb=1) == WS
    bwd = lambda cache, cb, flags=0, dh=FAKE: lib.mc_logprob_bwd_cached(
        FAKE, FAKE, FAKE, FAKE, FAKE, T, d, V, BF16, cache, cb, dh, FAKE, flags, FAKE_WS, need_b,
        None)
    assert bwd(None, need_c) == WS
    assert bwd(FAKE_WS, 0) == WS
    assert bwd(FAKE_WS, need_c, flags=8) == INVALID
    assert bwd(FAKE_WS, need_c, flags=12) == INVALID   # unknown bit beside a known one
    assert bwd(FAKE_WS, need_c, dh=FAKE + 4) == INVALID



def test_noalloc_loss_rejects_oversized_batches_on_the_host(lib):
    # the size check comes before any HIP call
    cap = lib.mc_rl_loss_noalloc_max_bytes()
    assert cap == 4 << 20
    assert lib.mc_rl_loss_workspace_size(0, 65536, 65536) <= cap
    p = binding.RLParams().to_c()
    o = binding.RLOutputsC(FAKE, FAKE, *([None] * (len(binding._OUT_FIELDS) - 2)))
    B = 1 << 20
    st = lib.mc_rl_loss_noalloc(FAKE, FAKE, None, None, FAKE, FAKE, FAKE, B, B, 1,
                                ctypes.byref(p), ctypes.byref(o), None)
    assert st == UNSUP
    bad = binding.RLParams(filter="none").to_c()
    bad.delta = -1.0
    assert lib.mc_rl_loss_noalloc(FAKE, FAKE, None, None, FAKE, FAKE, FAKE, 8, 2, 1,
                                  ctypes.byref(bad), ctypes.byref(o), None) == INVALID


def _consumer_source(names):
    """A program that takes the address of every declared entry point (so the
    link fails on any missing symbol) and prints the host-only queries."""
    refs = ",\n    ".join("(const void*)(size_t)&%s" % n for n in names)
    return f"""#include "mc.h"
#include <stdio.h>
#include <stddef.h>
int main(void) {{
  const void* volatile fns[] = {{
    {refs}
  }};
  size_t i, n = 0;
  for (i = 0; i < sizeof fns / sizeof fns[0]; ++i) n += fns[i] != NULL;
  printf("%zu\\n", n);
  printf("%s\\n", mc_version());
  printf("%s\\n", mc_status_string(MC_ERR_WORKSPACE));
  printf("%zu\\n", mc_rl_loss_noalloc_max_bytes());
  printf("%zu\\n", mc_logprob_bwd_workspace_size(16384, 4096, 151936, MC_BF16));
  printf("%zu\\n", mc_logprob_cache_size(16384, 4096, 151936, MC_BF16));
  return 0;
}}
"""


@pytest.mark.parametrize("lang", ["c99", "c++17"])
def test_header_builds_a_plain_consumer(lib, tmp_path, lang):
    """include/mc.h is a self-contained C header (and C++ through its
    extern "C" guard): a consumer built with warnings as errors links against
    libmc.so by name alone and sees the same values as the Python binding."""
    import shutil
    import subprocess
    cc = "gcc" if lang == "c99" else "g++"
    if shutil.which(cc) is None:
        pytest.skip(f"{cc} not installed")
    names = declared_functions()
    src = tmp_path / ("consumer.c" if lang == "c99" else "consumer.cpp")
    src.write_text(_consumer_source(names))
    exe = tmp_path / "consumer"
    libdir = os.path.dirname(binding.LIB_PATH)
    subprocess.run([cc, f"-std={lang}", "-Wall", "-Wextra", "-Werror", "-pedantic",
                    "-I", os.path.join(ROOT, "include"), str(src), "-L", libdir, "-lmc",
                    f"-Wl,-rpath,{libdir}", "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True,
                         timeout=60).stdout.split("\n")
    assert int(out[0]) == len(names)
    assert out[1] == binding.version()
    assert out[2] == "MC_ERR_WORKSPACE"
    assert int(out[3]) == lib.mc_rl_loss_noalloc_max_bytes()
    assert int(out[4]) == lib.mc_logprob_bwd_workspace_size(16384, 4096, 151936, BF16)
    assert int(out[5]) == lib.mc_logprob_cache_size(16384, 4096, 151936, BF16)
