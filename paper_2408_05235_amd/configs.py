"""The five synthetic workloads of the frequency-controller hot path.

Each workload is a batch of independent what-if scenarios.  A scenario is one
scoreboard (Sec. 4.2: per query the scheduling iteration, the input length and
the predicted generation length; Table 1), a KV-cache capacity (Sec. 4.3.2,
check 1), a per-token SLO (Sec. 4.3.2, checks 2 and 3; Sec. 5.1) and, in the
forest-bound workload, an engine size E (Table 1).  The performance model is a
seeded synthetic gradient-boosted forest over (frequency, KV blocks, batch
size[, engine size]) (Sec. 4.3.1).

Value ranges follow the paper's serving workload: prompts up to a few thousand
tokens, generations of tens to hundreds of tokens with a long tail (Sec. 3.4,
trace analysis), 16-token KV blocks, a few hundred to a few thousand future
iterations and per-token latencies of 10-50 ms (Sec. 5.2 reports 15-30 ms
TBT).  Fields marked ``proposed`` are not fixed by the workload description
and are chosen here.
"""

CONFIGS = [
    # c0: the small case the oracle finishes in milliseconds.
    dict(
        name="c0_single_scenario",
        n_scenarios=1,
        n_inflight=64,
        prompt=("uniform", 16, 1024),
        generated=("uniform", 0, 256),
        remaining=("uniform", 1, 512),
        queued=0,
        arrivals=None,
        block_tokens=16,
        kv_capacity=8192,
        batch_cap=None,
        horizon=512,
        n_freqs=17,
        # proposed: the model's batch range 0..256 (the other in-flight
        # workloads' size) rather than this board's 64, so that at the fixed
        # 20 ms SLO a frequency below the maximum passes
        forest=dict(n_trees=100, depth=6, n_features=3, leaves="profile",
                    base_score=40.0, batch_max=256),
        slo_ms=("fixed", 20.0),
        lost_scenario_prob=0.0,
        seed=1000,
    ),
    # c1: 1024 scenarios x 256 in-flight requests.
    dict(
        name="c1_1024x256",
        n_scenarios=1024,
        n_inflight=256,
        prompt=("uniform", 16, 4096),
        generated=("uniform", 0, 256),          # proposed
        remaining=("uniform", 1, 2048),
        queued=0,
        arrivals=None,
        block_tokens=16,
        kv_capacity=65536,
        batch_cap=None,
        horizon=2048,
        n_freqs=64,
        forest=dict(n_trees=500, depth=8, n_features=3, leaves="profile",
                    base_score=40.0, batch_max=256),
        slo_ms=("uniform_us", 10.0, 50.0),
        lost_scenario_prob=1.0 / 64,            # proposed
        seed=1001,
    ),
    # c2: long-context, 256 in-flight + 256 queued behind a batch cap.
    dict(
        name="c2_long_context_256x512",
        n_scenarios=256,
        n_inflight=256,                         # proposed split
        prompt=("lognormal", 8.0, 1.0, 1, 32768),
        generated=("uniform", 0, 256),          # proposed
        remaining=("uniform", 1, 4096),
        queued=256,                             # queued at iteration 0
        arrivals=None,
        block_tokens=16,
        kv_capacity=1 << 20,
        batch_cap=256,
        horizon=4096,
        n_freqs=32,
        forest=dict(n_trees=300, depth=8, n_features=3, leaves="profile",
                    base_score=40.0, batch_max=256),
        slo_ms=("uniform_us", 10.0, 50.0),      # proposed
        lost_scenario_prob=1.0 / 64,            # proposed
        seed=1002,
    ),
    # c3: forest-bound, 4 features including engine size.
    dict(
        name="c3_forest_bound_4096x128",
        n_scenarios=4096,
        n_inflight=128,
        prompt=("uniform", 16, 1024),           # proposed
        generated=("uniform", 0, 256),          # proposed
        remaining=("uniform", 1, 1024),         # proposed (fills the horizon)
        queued=0,
        arrivals=None,
        block_tokens=16,
        kv_capacity=65536,                      # proposed (never binds)
        batch_cap=None,
        horizon=1024,
        n_freqs=64,
        forest=dict(n_trees=2000, depth=10, n_features=4, leaves="normal",
                    leaf_sigma=0.1, base_score=40.0, batch_max=128),
        slo_ms=("uniform_us", 10.0, 50.0),      # proposed
        lost_scenario_prob=1.0 / 64,            # proposed
        seed=1003,
    ),
    # c4: 16384 scenarios, 256 in-flight + Poisson arrivals over the horizon.
    dict(
        name="c4_arrivals_16384x256",
        n_scenarios=16384,
        n_inflight=256,
        prompt=("uniform", 16, 2048),
        generated=("uniform", 0, 256),          # proposed
        remaining=("lognormal", 5.0, 1.2, 1, 8192),
        queued=0,
        arrivals=dict(rate=(0.5, 8.0),
                      length=("lognormal", 5.0, 1.2, 1, 8192),
                      prompt=("uniform", 16, 2048)),
        block_tokens=16,
        kv_capacity=131072,
        batch_cap=None,                         # proposed
        horizon=2048,
        n_freqs=48,
        forest=dict(n_trees=800, depth=8, n_features=3, leaves="profile",
                    base_score=40.0, batch_max=2048),
        slo_ms=("uniform_us", 10.0, 50.0),      # proposed
        lost_scenario_prob=1.0 / 64,            # proposed
        seed=1004,
    ),
]


def get_config(index_or_name):
    """Return a copy of one workload description, by index or by name."""
    if isinstance(index_or_name, int):
        return dict(CONFIGS[index_or_name])
    for cfg in CONFIGS:
        if cfg["name"] == index_or_name or cfg["name"].split("_")[0] == index_or_name:
            return dict(cfg)
    raise KeyError(index_or_name)
