"""The five verify-path workloads, with their shapes, distributions and seeds.

Model shapes follow the paper's target model, a Llama 3.1 8B-derived dense
decoder (paper §4 Experimental Setup): hidden 4096, FFN intermediate 14336,
fused QKV 6144 (32 query heads + 2x8 KV heads of 128), vocabulary 128256.
M = batch * (k + 1) draft-token rows per verify step (paper §3.1 EAGLE: the
target checks all drafted positions in one forward pass).
"""

from __future__ import annotations

HIDDEN = 4096
INTER = 14336
QKV_OUT = 6144
VOCAB = 128256

# Correlation coefficient c of the C4 logit generator, chosen so that greedy
# verification accepts a mean of 3.80 tokens per step (the paper's MGL for
# greedy EAGLE+FP8, Table 1).  Written by workloads/calibrate_c4.py, which
# calls only the CPU oracle.
C4_CORRELATION = 0.9995

# A 25-node draft tree in the style of an EAGLE top-k expansion: 4 candidates
# for the first new token, the higher-ranked branches expanded deeper (depth
# 6 along the top branch).  parent[n] of node n; -1 is the root.
TREE25 = (-1, -1, -1, -1,            # 0-3: first-position candidates
          0, 0, 0, 1, 1, 2, 3,       # 4-10
          4, 4, 4, 5, 7,             # 11-15
          11, 11, 12, 14,            # 16-19
          16, 16, 18,                # 20-22
          20, 20)                    # 23-24

# The four linears of one decoder layer: (name, N, K) with W [N,K].
LAYER_LINEARS = (
    ("qkv", QKV_OUT, HIDDEN),
    ("o", HIDDEN, HIDDEN),
    ("gate_up", 2 * INTER, HIDDEN),
    ("down", HIDDEN, INTER),
)

CONFIGS = {
    "C1": dict(
        desc="tiny verify step: B=2, k=3 -> M=8; one FP8 linear 512->1024; accept over V=256",
        B=2, k=3, M=8, K=512, N=1024, V=256,
        act_outlier_frac=0.01, act_outlier_scale=20.0, w_std=0.02,
        logit_std=2.0, temperature=0.7, seed=0,
    ),
    "C2": dict(
        desc="one decoder layer's verify linears at B=16, k=4 -> M=80, hidden 4096",
        B=16, k=4, M=80, linears=LAYER_LINEARS,
        act_outlier_frac=0.005, act_outlier_scale=30.0, w_std=0.02, seed=1,
    ),
    "C3": dict(
        desc="one decoder layer's verify linears at serving batch B=64, k=4 -> M=320, "
             "SiLU-gated FFN re-quantized into the down projection, bf16 output",
        B=64, k=4, M=320, linears=LAYER_LINEARS,
        act_outlier_frac=0.005, act_outlier_scale=30.0, w_std=0.02, seed=2,
    ),
    "C4": dict(
        desc="acceptance at full vocabulary: B=64, k=4, V=128256, greedy and T=0.7",
        B=64, k=4, V=VOCAB, logit_std=3.0, rank=8, temperature=0.7,
        seed=7, draft_seed=8, uniform_seed=7,
    ),
    "CALSTUDY": dict(
        desc="static per-tensor calibration study: clip rate of an 8192-token in-domain-like test set "
             "against scales calibrated on 32..2048 tokens of a public-like, an in-domain-like and a "
             "mixed synthetic set (hidden size 4096)",
        K=HIDDEN, lengths=(32, 64, 128, 256, 512, 1024, 2048), test_tokens=8192,
        public_outlier_frac=0.005, public_outlier_scale=30.0, indomain_df=3.0, seed=21,
    ),
    "DRAFT": dict(
        desc="FP8 linears of the EAGLE-style drafter (the feature fc 8192->4096 plus one "
             "Llama-3.1-8B-shaped decoder layer, about 250M parameters) for one draft step of "
             "B=64 sequences (M=64), static per-tensor activation scales from min-max calibration",
        B=64, M=64, linears=(("fc", HIDDEN, 2 * HIDDEN),) + LAYER_LINEARS, n_calib=8,
        act_outlier_frac=0.005, act_outlier_scale=30.0, w_std=0.02, seed=13,
    ),
    "KV": dict(
        desc="FP8 KV-cache write of the verify step's new tokens: B=64, k=4 -> T=320 tokens, "
             "8 KV heads of 128 (Llama 3.1 8B), paged cache with 16-token blocks, "
             "contexts of 512..4096 tokens per sequence",
        B=64, k=4, T=320, H=8, D=128, block_size=16, ctx_min=512, ctx_max=4096,
        key_outlier_frac=0.01, key_outlier_scale=20.0, seed=11,
    ),
    "C5": dict(
        desc="long-prompt prefill/calibration: M=4096, 4096->14336 and 14336->4096, "
             "Student-t(3) activations, static per-tensor vs dynamic per-token scales",
        M=4096, K1=HIDDEN, N1=INTER, K2=INTER, N2=HIDDEN, df=3.0,
        n_calib=32, w_std=0.02, seed=5,
    ),
}
