"""ctypes binding of libmc.so (declared in include/mc.h).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  torch provides device memory (outputs and workspaces) and the
current stream; no torch operator touches the data.  If the library is
missing the binding raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libmc.so")

MC_OK, MC_ERR_INVALID_ARG, MC_ERR_UNSUPPORTED, MC_ERR_WORKSPACE, MC_ERR_HIP = range(5)
MC_F32, MC_BF16 = 0, 1
MC_FILTER = {"none": 0, "vanilla": 1, "mirrorpop": 2}
MC_TOKEN = {"none": 0, "tis": 1, "icepop": 2}
MC_BWD_ACCUMULATE_DHIDDEN = 1
MC_BWD_ACCUMULATE_DWEIGHT = 2
MC_BWD_SKIP_DEAD_TOKENS = 4

_c_i64, _c_i32, _c_sz, _vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t, ctypes.c_void_p


class RLParamsC(ctypes.Structure):
    _fields_ = [("eps_low", ctypes.c_float), ("eps_high", ctypes.c_float),
                ("delta", ctypes.c_float), ("adv_eps", ctypes.c_float),
                ("std_ddof", ctypes.c_int32), ("filter", ctypes.c_int32),
                ("kl_beta", ctypes.c_float), ("token_mode", ctypes.c_int32),
                ("tis_cap", ctypes.c_float), ("icepop_lo", ctypes.c_float),
                ("icepop_hi", ctypes.c_float)]


_OUT_FIELDS = ("loss", "dlogp", "seq_mask", "seq_len", "n_valid", "adv", "stat_abs",
               "stat_signed", "clip_frac", "error_flag", "kl", "token_frac")


class RLOutputsC(ctypes.Structure):
    _fields_ = [(n, _vp) for n in _OUT_FIELDS]


class KernelTimeC(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double), ("total_flops", ctypes.c_double),
                ("total_bytes", ctypes.c_double)]


@dataclasses.dataclass
class RLParams:
    eps_low: float = 0.2
    eps_high: float = 0.2
    delta: float = 0.1
    adv_eps: float = 1e-6
    std_ddof: int = 0
    filter: str = "mirrorpop"
    kl_beta: float = 0.0
    token_mode: str = "none"
    tis_cap: float = 2.0
    icepop_lo: float = 0.5
    icepop_hi: float = 2.0

    def to_c(self) -> RLParamsC:
        return RLParamsC(self.eps_low, self.eps_high, self.delta, self.adv_eps,
                         int(self.std_ddof), MC_FILTER[self.filter], self.kl_beta,
                         MC_TOKEN[self.token_mode], self.tis_cap, self.icepop_lo,
                         self.icepop_hi)


class MCError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)}")
        self.status = status


_LIB = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libmc.so (once).  Raises if it has not been built."""
    global _LIB
    if _LIB is not None and path == LIB_PATH:
        return _LIB
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with "
                          "`python -m paper_2606_04847_amd.build`")
    lib = ctypes.CDLL(path)
    lib.mc_status_string.restype = ctypes.c_char_p
    lib.mc_status_string.argtypes = [ctypes.c_int]
    lib.mc_version.restype = ctypes.c_char_p
    lib.mc_version.argtypes = []
    for name in ("mc_logprob_fwd_workspace_size", "mc_logprob_bwd_workspace_size",
                 "mc_logprob_cache_size", "mc_logprob_bwd_cached_workspace_size"):
        f = getattr(lib, name)
        f.restype = _c_sz
        f.argtypes = [_c_i64, _c_i64, _c_i64, ctypes.c_int]
    lib.mc_rl_loss_workspace_size.restype = _c_sz
    lib.mc_rl_loss_workspace_size.argtypes = [_c_i64, _c_i32, _c_i32]
    lib.mc_logprob_fwd.restype = ctypes.c_int
    lib.mc_logprob_fwd.argtypes = [_vp, _vp, _vp, _c_i64, _c_i64, _c_i64, ctypes.c_int,
                                   _vp, _vp, _vp, _vp, _c_sz, _vp]
    lib.mc_logprob_fwd_shard.restype = ctypes.c_int
    lib.mc_logprob_fwd_shard.argtypes = [_vp, _vp, _vp, _c_i64, _c_i64, _c_i64, _c_i64, _c_i64,
                                         ctypes.c_int, _vp, _vp, _c_sz, _vp]
    lib.mc_logprob_merge_shards.restype = ctypes.c_int
    lib.mc_logprob_merge_shards.argtypes = [_vp, _c_i32, _vp, _c_i64, _c_i64, _vp, _vp, _vp, _vp]
    lib.mc_logprob_bwd.restype = ctypes.c_int
    lib.mc_logprob_bwd.argtypes = [_vp, _vp, _vp, _vp, _vp, _c_i64, _c_i64, _c_i64,
                                   ctypes.c_int, _vp, _vp, _c_i32, _vp, _c_sz, _vp]
    lib.mc_logprob_fwd_cached.restype = ctypes.c_int
    lib.mc_logprob_fwd_cached.argtypes = [_vp, _vp, _vp, _c_i64, _c_i64, _c_i64, ctypes.c_int,
                                          _vp, _vp, _vp, _vp, _c_sz, _vp, _c_sz, _vp]
    lib.mc_logprob_bwd_cached.restype = ctypes.c_int
    lib.mc_logprob_bwd_cached.argtypes = [_vp, _vp, _vp, _vp, _vp, _c_i64, _c_i64, _c_i64,
                                          ctypes.c_int, _vp, _c_sz, _vp, _vp, _c_i32, _vp,
                                          _c_sz, _vp]
    lib.mc_logprob_bwd_shard.restype = ctypes.c_int
    lib.mc_logprob_bwd_shard.argtypes = [_vp, _vp, _vp, _vp, _vp, _c_i64, _c_i64, _c_i64,
                                         _c_i64, _c_i64, ctypes.c_int, _vp, _vp, _c_i32, _vp,
                                         _c_sz, _vp]
    lib.mc_rl_loss.restype = ctypes.c_int
    lib.mc_rl_loss.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _c_i64, _c_i32, _c_i32,
                               ctypes.POINTER(RLParamsC), ctypes.POINTER(RLOutputsC),
                               _vp, _c_sz, _vp]
    lib.mc_rl_loss_noalloc.restype = ctypes.c_int
    lib.mc_rl_loss_noalloc.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _c_i64, _c_i32,
                                       _c_i32, ctypes.POINTER(RLParamsC),
                                       ctypes.POINTER(RLOutputsC), _vp]
    lib.mc_rl_loss_noalloc_max_bytes.restype = _c_sz
    lib.mc_rl_loss_noalloc_max_bytes.argtypes = []
    lib.mc_primeecho_rewards.restype = ctypes.c_int
    lib.mc_primeecho_rewards.argtypes = [_vp, _vp, _vp, _c_i32, _c_i32, ctypes.c_float,
                                         ctypes.c_float, ctypes.c_float, _vp, _vp]
    lib.mc_check_packing.restype = ctypes.c_int
    lib.mc_check_packing.argtypes = [_vp, _c_i32, _vp, _c_i32, _c_i64]
    lib.mc_profiler_enable.restype = None
    lib.mc_profiler_enable.argtypes = [_c_i32]
    lib.mc_profiler_reset.restype = None
    lib.mc_profiler_reset.argtypes = []
    lib.mc_profiler_read.restype = _c_i32
    lib.mc_profiler_read.argtypes = [ctypes.POINTER(KernelTimeC), _c_i32]
    if path == LIB_PATH:
        _LIB = lib
    return lib


def status_string(status: int) -> str:
    return load_library().mc_status_string(status).decode()


def version() -> str:
    return load_library().mc_version().decode()


# ---------------------------------------------------------------------------
# torch-facing helpers (device memory and streams only)
# ---------------------------------------------------------------------------
def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return MC_BF16
    if t.dtype == torch.float32:
        return MC_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _check(status, what):
    if status != MC_OK:
        raise MCError(status, what)


def _workspace(nbytes, device, workspace=None, owned=None):
    """The caller's workspace when it is large enough, else a new one (added
    to `owned`, the list of tensors this wrapper allocated)."""
    torch = _torch()
    if nbytes == 0:
        return None, 0
    if workspace is not None and workspace.numel() >= nbytes:
        return workspace, workspace.numel()
    ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    if owned is not None:
        owned.append(ws)
    return ws, nbytes


def _new(owned, *shape, dtype, device):
    """An uninitialised device tensor allocated by a wrapper (kept in `owned`)."""
    t = _torch().empty(*shape, dtype=dtype, device=device)
    owned.append(t)
    return t


def _keep_alive(stream, *tensors):
    """Memory a wrapper allocated on the current stream but handed to kernels
    enqueued on another stream: record that stream on it, so the caching
    allocator does not reuse it before that stream's work is done."""
    if stream is None:
        return
    for t in tensors:
        if t is not None:
            t.record_stream(stream)


def _need(cond, msg):
    if not cond:
        raise ValueError(msg)


def logprob_fwd(hidden, weight, targets, *, logp=None, lse=None, entropy=None,
                with_entropy=False, workspace=None, stream=None):
    """Per-token log-prob over the full vocabulary (see mc_logprob_fwd).

    hidden [T,d] and weight [V,d] bf16 or fp32 (same dtype), targets [T] int64,
    all on one GPU.  Returns (logp, lse), fp32 [T], or (logp, lse, entropy)
    when with_entropy is set."""
    torch = _torch()
    lib = load_library()
    _need(hidden.is_cuda and weight.is_cuda and targets.is_cuda, "tensors must be on the GPU")
    _need(hidden.dtype == weight.dtype, "hidden and weight dtypes differ")
    _need(targets.dtype == torch.int64, "targets must be int64")
    _need(hidden.is_contiguous() and weight.is_contiguous() and targets.is_contiguous(),
          "tensors must be contiguous")
    T, d = hidden.shape
    V = weight.shape[0]
    _need(weight.shape[1] == d and targets.shape == (T,), "shape mismatch")
    dt = _dtype_code(hidden)
    dev = hidden.device
    owned = []
    f32 = torch.float32
    logp = _new(owned, T, dtype=f32, device=dev) if logp is None else logp
    lse = _new(owned, T, dtype=f32, device=dev) if lse is None else lse
    if with_entropy and entropy is None:
        entropy = _new(owned, T, dtype=f32, device=dev)
    need = lib.mc_logprob_fwd_workspace_size(T, d, V, dt)
    ws, nbytes = _workspace(need, dev, workspace, owned)
    _check(lib.mc_logprob_fwd(_ptr(hidden), _ptr(weight), _ptr(targets), T, d, V, dt,
                              _ptr(logp), _ptr(lse), _ptr(entropy), _ptr(ws), nbytes,
                              _stream(stream)), "mc_logprob_fwd")
    _keep_alive(stream, *owned)
    return (logp, lse, entropy) if entropy is not None else (logp, lse)


def logprob_fwd_shard(hidden, weight_shard, targets, v_offset, V_total, *, partial=None,
                      workspace=None, stream=None):
    """Partial forward on a vocabulary shard (see mc_logprob_fwd_shard).
    Returns partial [4, T] fp32: (max, sum exp, sum exp*z, target logit or -inf)."""
    torch = _torch()
    lib = load_library()
    T, d = hidden.shape
    Vs = weight_shard.shape[0]
    _need(hidden.dtype == weight_shard.dtype and targets.dtype == torch.int64, "dtypes")
    for t in (hidden, weight_shard, targets):
        _need(t.is_cuda and t.is_contiguous(), "contiguous GPU tensors")
    dt = _dtype_code(hidden)
    dev = hidden.device
    owned = []
    if partial is None:
        partial = _new(owned, 4, T, dtype=torch.float32, device=dev)
    need = lib.mc_logprob_fwd_workspace_size(T, d, Vs, dt)
    ws, nbytes = _workspace(need, dev, workspace, owned)
    _check(lib.mc_logprob_fwd_shard(_ptr(hidden), _ptr(weight_shard), _ptr(targets), T, d, Vs,
                                    int(v_offset), int(V_total), dt, _ptr(partial), _ptr(ws),
                                    nbytes, _stream(stream)), "mc_logprob_fwd_shard")
    _keep_alive(stream, *owned)
    return partial


def logprob_merge_shards(partials, targets, V_total, *, with_entropy=True, stream=None):
    """Fold partials [S, 4, T] (shard order) into (logp, lse, entropy)."""
    torch = _torch()
    lib = load_library()
    S, four, T = partials.shape
    _need(four == 4 and partials.dtype == torch.float32 and partials.is_contiguous(),
          "partials [S, 4, T] fp32")
    dev = partials.device
    owned = []
    logp = _new(owned, T, dtype=torch.float32, device=dev)
    lse = _new(owned, T, dtype=torch.float32, device=dev)
    ent = _new(owned, T, dtype=torch.float32, device=dev) if with_entropy else None
    _check(lib.mc_logprob_merge_shards(_ptr(partials), S, _ptr(targets), T, int(V_total),
                                       _ptr(logp), _ptr(lse), _ptr(ent), _stream(stream)),
           "mc_logprob_merge_shards")
    _keep_alive(stream, *owned)
    return logp, lse, ent


def logprob_bwd_shard(hidden, weight_shard, targets, lse, dlogp, v_offset, V_total, *,
                      dhidden=None, dweight=None, need_dhidden=True, need_dweight=True,
                      skip_dead_tokens=False, workspace=None, stream=None):
    """Backward on a vocabulary shard (see mc_logprob_bwd_shard).  Returns
    (this shard's part of dhidden, the shard's rows of dW)."""
    torch = _torch()
    lib = load_library()
    T, d = hidden.shape
    Vs = weight_shard.shape[0]
    dt = _dtype_code(hidden)
    dev = hidden.device
    owned = []
    if need_dhidden and dhidden is None:
        dhidden = _new(owned, T, d, dtype=torch.float32, device=dev)
    if need_dweight and dweight is None:
        dweight = _new(owned, Vs, d, dtype=torch.float32, device=dev)
    need = lib.mc_logprob_bwd_workspace_size(T, d, Vs, dt)
    ws, nbytes = _workspace(need, dev, workspace, owned)
    _check(lib.mc_logprob_bwd_shard(_ptr(hidden), _ptr(weight_shard), _ptr(targets), _ptr(lse),
                                    _ptr(dlogp), T, d, Vs, int(v_offset), int(V_total), dt,
                                    _ptr(dhidden if need_dhidden else None),
                                    _ptr(dweight if need_dweight else None),
                                    MC_BWD_SKIP_DEAD_TOKENS if skip_dead_tokens else 0, _ptr(ws),
                                    nbytes, _stream(stream)), "mc_logprob_bwd_shard")
    _keep_alive(stream, *owned)
    return (dhidden if need_dhidden else None), (dweight if need_dweight else None)


def primeecho_rewards(scores, success=None, n_turns=None, *, alpha=0.75, beta1=0.0, beta2=0.0,
                      stream=None):
    """PrimeEcho trajectory rewards (see mc_primeecho_rewards): scores [B, Kmax]
    fp32, success [B, Kmax] uint8, n_turns [B] int32.  Returns rewards [B]."""
    torch = _torch()
    lib = load_library()
    B, K = scores.shape
    _need(scores.dtype == torch.float32 and scores.is_cuda and scores.is_contiguous(),
          "scores fp32 [B, Kmax] on the GPU")
    _need(success is None or (success.dtype == torch.uint8 and success.shape == (B, K)),
          "success uint8 [B, Kmax]")
    _need(n_turns is None or (n_turns.dtype == torch.int32 and n_turns.shape == (B,)),
          "n_turns int32 [B]")
    owned = []
    out = _new(owned, B, dtype=torch.float32, device=scores.device)
    _check(lib.mc_primeecho_rewards(_ptr(scores), _ptr(success), _ptr(n_turns), B, K,
                                    float(alpha), float(beta1), float(beta2), _ptr(out),
                                    _stream(stream)), "mc_primeecho_rewards")
    _keep_alive(stream, *owned)
    return out


def logprob_bwd(hidden, weight, targets, lse, dlogp, *, dhidden=None, dweight=None,
                need_dhidden=True, need_dweight=True, accumulate_dhidden=False,
                accumulate_dweight=False, skip_dead_tokens=False, workspace=None, stream=None):
    """Gradients of sum_t dlogp_t logp_t (see mc_logprob_bwd).  skip_dead_tokens:
    MC_BWD_SKIP_DEAD_TOKENS.  Returns (dhidden [T,d] fp32 or None, dweight
    [V,d] fp32 or None)."""
    torch = _torch()
    lib = load_library()
    T, d = hidden.shape
    V = weight.shape[0]
    _need(hidden.dtype == weight.dtype, "hidden and weight dtypes differ")
    _need(targets.dtype == torch.int64 and lse.dtype == torch.float32
          and dlogp.dtype == torch.float32, "targets int64, lse/dlogp fp32")
    for t in (hidden, weight, targets, lse, dlogp):
        _need(t.is_cuda and t.is_contiguous(), "tensors must be contiguous on the GPU")
    _need(lse.shape == (T,) and dlogp.shape == (T,) and targets.shape == (T,), "shape mismatch")
    dt = _dtype_code(hidden)
    dev = hidden.device
    owned = []
    if need_dhidden and dhidden is None:
        dhidden = _new(owned, T, d, dtype=torch.float32, device=dev)
    if need_dweight and dweight is None:
        dweight = _new(owned, V, d, dtype=torch.float32, device=dev)
    if not need_dhidden:
        dhidden = None
    if not need_dweight:
        dweight = None
    flags = ((MC_BWD_ACCUMULATE_DHIDDEN if accumulate_dhidden else 0)
             | (MC_BWD_ACCUMULATE_DWEIGHT if accumulate_dweight else 0)
             | (MC_BWD_SKIP_DEAD_TOKENS if skip_dead_tokens else 0))
    need = lib.mc_logprob_bwd_workspace_size(T, d, V, dt)
    ws, nbytes = _workspace(need, dev, workspace, owned)
    _check(lib.mc_logprob_bwd(_ptr(hidden), _ptr(weight), _ptr(targets), _ptr(lse), _ptr(dlogp),
                              T, d, V, dt, _ptr(dhidden), _ptr(dweight), flags, _ptr(ws),
                              nbytes, _stream(stream)), "mc_logprob_bwd")
    _keep_alive(stream, *owned)
    return dhidden, dweight


def softmax_cache(hidden, weight):
    """An uninitialised softmax cache for hidden [T,d] and weight [V,d] (see
    mc_logprob_fwd_cached): a uint8 device tensor of mc_logprob_cache_size bytes."""
    torch = _torch()
    lib = load_library()
    T, d = hidden.shape
    V = weight.shape[0]
    n = lib.mc_logprob_cache_size(T, d, V, _dtype_code(hidden))
    return torch.empty(max(int(n), 1), dtype=torch.uint8, device=hidden.device)


def logprob_fwd_cached(hidden, weight, targets, cache, *, logp=None, lse=None, entropy=None,
                       with_entropy=False, workspace=None, stream=None):
    """mc_logprob_fwd_cached: logprob_fwd that also fills `cache` (from
    softmax_cache) for one later logprob_bwd_cached call."""
    torch = _torch()
    lib = load_library()
    _need(hidden.is_cuda and weight.is_cuda and targets.is_cuda, "tensors must be on the GPU")
    _need(hidden.dtype == weight.dtype, "hidden and weight dtypes differ")
    _need(targets.dtype == torch.int64, "targets must be int64")
    _need(hidden.is_contiguous() and weight.is_contiguous() and targets.is_contiguous(),
          "tensors must be contiguous")
    T, d = hidden.shape
    V = weight.shape[0]
    _need(weight.shape[1] == d and targets.shape == (T,), "shape mismatch")
    dt = _dtype_code(hidden)
    dev = hidden.device
    owned = []
    f32 = torch.float32
    logp = _new(owned, T, dtype=f32, device=dev) if logp is None else logp
    lse = _new(owned, T, dtype=f32, device=dev) if lse is None else lse
    if with_entropy and entropy is None:
        entropy = _new(owned, T, dtype=f32, device=dev)
    need = lib.mc_logprob_fwd_workspace_size(T, d, V, dt)
    ws, nbytes = _workspace(need, dev, workspace, owned)
    _check(lib.mc_logprob_fwd_cached(_ptr(hidden), _ptr(weight), _ptr(targets), T, d, V, dt,
                                     _ptr(logp), _ptr(lse), _ptr(entropy), _ptr(cache),
                                     cache.numel(), _ptr(ws), nbytes, _stream(stream)),
           "mc_logprob_fwd_cached")
    _keep_alive(stream, *owned)
    return (logp, lse, entropy) if entropy is not None else (logp, lse)


def logprob_bwd_cached(hidden, weight, targets, lse, dlogp, cache, *, dhidden=None,
                       dweight=None, need_dhidden=True, need_dweight=True,
                       accumulate_dhidden=False, accumulate_dweight=False,
                       skip_dead_tokens=False, workspace=None, stream=None):
    """mc_logprob_bwd_cached: logprob_bwd from the cache the forward filled
    (read only)."""
    torch = _torch()
    lib = load_library()
    T, d = hidden.shape
    V = weight.shape[0]
    _need(hidden.dtype == weight.dtype, "hidden and weight dtypes differ")
    _need(targets.dtype == torch.int64 and lse.dtype == torch.float32
          and dlogp.dtype == torch.float32, "targets int64, lse/dlogp fp32")
    for t in (hidden, weight, targets, lse, dlogp, cache):
        _need(t.is_cuda and t.is_contiguous(), "tensors must be contiguous on the GPU")
    _need(lse.shape == (T,) and dlogp.shape == (T,) and targets.shape == (T,), "shape mismatch")
    dt = _dtype_code(hidden)
    dev = hidden.device
    owned = []
    if need_dhidden and dhidden is None:
        dhidden = _new(owned, T, d, dtype=torch.float32, device=dev)
    if need_dweight and dweight is None:
        dweight = _new(owned, V, d, dtype=torch.float32, device=dev)
    if not need_dhidden:
        dhidden = None
    if not need_dweight:
        dweight = None
    flags = ((MC_BWD_ACCUMULATE_DHIDDEN if accumulate_dhidden else 0)
             | (MC_BWD_ACCUMULATE_DWEIGHT if accumulate_dweight else 0)
             | (MC_BWD_SKIP_DEAD_TOKENS if skip_dead_tokens else 0))
    need = lib.mc_logprob_bwd_cached_workspace_size(T, d, V, dt)
    ws, nbytes = _workspace(need, dev, workspace, owned)
    _check(lib.mc_logprob_bwd_cached(_ptr(hidden), _ptr(weight), _ptr(targets), _ptr(lse),
                                     _ptr(dlogp), T, d, V, dt, _ptr(cache), cache.numel(),
                                     _ptr(dhidden), _ptr(dweight), flags, _ptr(ws), nbytes,
                                     _stream(stream)), "mc_logprob_bwd_cached")
    _keep_alive(stream, *owned)
    return dhidden, dweight


def rl_loss(logp, logp_rollout, loss_mask, cu_seqlens, cu_groups, rewards,
            params: RLParams | None = None, *, logp_ref=None, workspace=None, stream=None,
            out=None, noalloc=False):
    """RL objective over a packed batch (see mc_rl_loss).  Returns a dict of
    device tensors: loss, dlogp, seq_mask, seq_len, n_valid, adv, stat_abs,
    stat_signed, clip_frac, error_flag, kl, token_frac (`out` may supply
    them).  noalloc=True calls mc_rl_loss_noalloc, which takes no workspace
    (with `out` given, this wrapper allocates nothing either)."""
    torch = _torch()
    lib = load_library()
    p = params or RLParams()
    T = logp.shape[0]
    B = cu_seqlens.shape[0] - 1
    NG = cu_groups.shape[0] - 1
    _need(logp.dtype == torch.float32 and logp_rollout.dtype == torch.float32, "fp32 log-probs")
    _need(cu_seqlens.dtype == torch.int32 and cu_groups.dtype == torch.int32, "int32 offsets")
    _need(rewards.dtype == torch.float32 and rewards.shape == (B,), "rewards fp32 [B]")
    _need(loss_mask is None or (loss_mask.dtype == torch.uint8 and loss_mask.shape == (T,)),
          "loss_mask uint8 [T]")
    _need(logp_ref is None or (logp_ref.dtype == torch.float32 and logp_ref.shape == (T,)),
          "logp_ref fp32 [T]")
    for t in (logp, logp_rollout, logp_ref, cu_seqlens, cu_groups, rewards, loss_mask):
        _need(t is None or (t.is_cuda and t.is_contiguous()), "contiguous GPU tensors")
    dev = logp.device
    given = out
    out = dict(
        loss=torch.empty(1, dtype=torch.float32, device=dev),
        dlogp=torch.empty(T, dtype=torch.float32, device=dev),
        seq_mask=torch.empty(B, dtype=torch.uint8, device=dev),
        seq_len=torch.empty(B, dtype=torch.int32, device=dev),
        n_valid=torch.empty(1, dtype=torch.int64, device=dev),
        adv=torch.empty(B, dtype=torch.float32, device=dev),
        stat_abs=torch.empty(B, dtype=torch.float32, device=dev),
        stat_signed=torch.empty(B, dtype=torch.float32, device=dev),
        clip_frac=torch.empty(1, dtype=torch.float32, device=dev),
        error_flag=torch.empty(1, dtype=torch.int32, device=dev),
        kl=torch.empty(1, dtype=torch.float32, device=dev),
        token_frac=torch.empty(1, dtype=torch.float32, device=dev),
    ) if given is None else given
    oc = RLOutputsC(*[out[k].data_ptr() if out.get(k) is not None and out[k].numel() else None
                      for k in _OUT_FIELDS])
    pc = p.to_c()
    owned = [] if given is not None else list(out.values())
    if noalloc:
        _check(lib.mc_rl_loss_noalloc(_ptr(logp), _ptr(logp_rollout), _ptr(logp_ref),
                                      _ptr(loss_mask), _ptr(cu_seqlens), _ptr(cu_groups),
                                      _ptr(rewards), T, B, NG, ctypes.byref(pc),
                                      ctypes.byref(oc), _stream(stream)), "mc_rl_loss_noalloc")
    else:
        need = lib.mc_rl_loss_workspace_size(T, B, NG)
        ws, nbytes = _workspace(need, dev, workspace, owned)
        _check(lib.mc_rl_loss(_ptr(logp), _ptr(logp_rollout), _ptr(logp_ref), _ptr(loss_mask),
                              _ptr(cu_seqlens),
                              _ptr(cu_groups), _ptr(rewards), T, B, NG, ctypes.byref(pc),
                              ctypes.byref(oc), _ptr(ws), nbytes, _stream(stream)), "mc_rl_loss")
    _keep_alive(stream, *owned)
    return out


def check_packing(cu_seqlens_host, cu_groups_host, T: int) -> bool:
    """Host-side validation of packing metadata (numpy int32 arrays)."""
    import numpy as np
    lib = load_library()
    cu = np.ascontiguousarray(cu_seqlens_host, dtype=np.int32)
    cg = np.ascontiguousarray(cu_groups_host, dtype=np.int32)
    st = lib.mc_check_packing(cu.ctypes.data_as(_vp), len(cu) - 1, cg.ctypes.data_as(_vp),
                              len(cg) - 1, int(T))
    return st == MC_OK


def profiler_enable(on: bool = True) -> None:
    """Bracket every later launch with hipEvents on its stream (mc_profiler_*)."""
    load_library().mc_profiler_enable(1 if on else 0)


def profiler_reset() -> None:
    load_library().mc_profiler_reset()


def profiler_read() -> dict:
    """Per-kernel totals: {name: dict(launches, ms, flops, bytes)}."""
    lib = load_library()
    n = lib.mc_profiler_read(None, 0)
    arr = (KernelTimeC * max(n, 1))()
    n = lib.mc_profiler_read(arr, n)
    return {arr[i].name.decode(): dict(launches=int(arr[i].launches), ms=arr[i].total_ms,
                                       flops=arr[i].total_flops, bytes=arr[i].total_bytes)
            for i in range(n)}
