"""MI355X-native fused RL log-prob path (hand-written HIP kernels for gfx950
behind a C ABI, include/mc.h).

    from paper_2606_04847_amd import logprob_fwd, rl_loss, logprob_bwd
"""
from .binding import (  # noqa: F401
    LIB_PATH,
    MCError,
    RLParams,
    check_packing,
    load_library,
    logprob_bwd,
    logprob_bwd_cached,
    logprob_fwd_cached,
    softmax_cache,
    logprob_bwd_shard,
    logprob_fwd,
    logprob_fwd_shard,
    logprob_merge_shards,
    primeecho_rewards,
    profiler_enable,
    profiler_read,
    profiler_reset,
    rl_loss,
    status_string,
    version,
)
