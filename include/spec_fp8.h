/*
 * spec_fp8.h -- C ABI of libspecfp8.so, the FP8 speculative-decoding verify
 * path for AMD Instinct MI355X (gfx950).
 *
 * The verify step of speculative decoding (paper section 3.1, EAGLE): a draft
 * model proposes k tokens per sequence, the target model scores all k+1
 * positions of B sequences in one forward pass whose linear layers run as
 * FP8 E4M3 W8A8 (paper section 3.2, FP8 Post-Training Quantization) over
 * M = B*(k+1) rows, and an acceptance test keeps the longest agreeing prefix
 * plus one resampled or bonus token.
 *
 * Conventions shared by every entry point:
 *  - Every buffer argument is DEVICE memory owned by the caller, except where
 *    a comment says otherwise.  The library never allocates, frees or
 *    synchronizes; it validates arguments on the host and then enqueues work
 *    asynchronously on `stream` (a hipStream_t passed as void*; NULL means the
 *    default stream).  Outputs are valid once that stream has reached the
 *    enqueued work.
 *  - All argument errors are detected on the host, before any HIP call, and
 *    returned as a status; nothing is enqueued then.  A failed kernel launch
 *    returns SPEC_ERR_HIP and records the hipError_t for spec_last_hip_error().
 *  - Matrices are row-major; `ld_*` is the row stride in elements.
 *  - bf16 tensors are raw 16-bit bfloat16 bit patterns (uint16_t storage).
 *  - FP8 tensors are OCP E4M3 ("E4M3FN") bytes: bias 7, no infinities, NaN is
 *    S.1111.111, largest finite magnitude 448.
 *  - Calls are reentrant; the only global state is a thread-local copy of the
 *    last HIP error.  Calls that share output or workspace buffers must not
 *    overlap on different streams.
 */
#ifndef SPEC_FP8_H
#define SPEC_FP8_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SPEC_OK = 0,
    SPEC_ERR_NULL = 1,         /* a required pointer is NULL                         */
    SPEC_ERR_SHAPE = 2,        /* a size is negative/zero where not allowed, ld < cols */
    SPEC_ERR_UNSUPPORTED = 3,  /* valid but outside the supported fast path          */
    SPEC_ERR_ENUM = 4,         /* an enum argument holds an unknown value            */
    SPEC_ERR_ALIGN = 5,        /* pointer or stride misaligned for vector access     */
    SPEC_ERR_WORKSPACE = 6,    /* workspace missing or smaller than required         */
    SPEC_ERR_HIP = 7,          /* a HIP launch failed (see spec_last_hip_error)      */
    SPEC_ERR_VALUE = 8,        /* a scalar argument is out of range (e.g. temperature) */
    SPEC_ERR_SCRATCH = 9       /* the call needs more than the library's fixed scratch */
} spec_status;

typedef enum {
    SPEC_SCALE_PER_ROW = 0,    /* dynamic: one scale per row (per token for activations,
                                  per output channel for weights W[N,K])              */
    SPEC_SCALE_PER_TENSOR = 1, /* static: one fp32 scale for the whole tensor         */
    SPEC_SCALE_CALIBRATE = 2   /* spec_fp8_quantize only: fold the tensor's scale into a
                                  running static scale (min-max calibration)          */
} spec_scale_mode;

typedef enum {
    SPEC_QIN_BF16 = 0,         /* quantize x itself                                   */
    SPEC_QIN_SILU_MUL_BF16 = 1 /* quantize h = bf16(silu(x[:, c]) * x[:, cols + c])   */
} spec_quant_input;

typedef enum {
    SPEC_OUT_BF16 = 0,         /* bf16, round-to-nearest-even of the fp32 result       */
    SPEC_OUT_F32 = 1
} spec_out_dtype;

/*
 * spec_fp8_quantize -- rows of bf16 values to E4M3 codes with fp32 scales.
 *
 * The paper quantizes activations and weights to E4M3 with min-max scales
 * (section 3.2); E4M3 is symmetric with no zero point, so the scale of a
 * range with largest magnitude amax is amax / 448.  For every row r:
 *
 *   v[c]  = x[r,c]                                   (in_kind = SPEC_QIN_BF16)
 *         = bf16(silu(x[r,c]) * x[r,cols+c])         (SPEC_QIN_SILU_MUL_BF16: x is
 *           [rows, 2*cols], gate columns first, then up; the gated FFN of the
 *           Llama-family target model, section 4)
 *   PER_ROW:    s[r] = max(fl32(max_c |v[c]| / 448), 2^-100); scales[r] = s[r]   (written)
 *   PER_TENSOR: s[r] = scales[0]                                               (read)
 *   q[r,c] = E4M3(fl32(v[c] * fl32(1 / s[r])))
 *   CALIBRATE:  scales[0] = max(scales[0], max_r s[r]) with s[r] as for PER_ROW;
 *               nothing else is written (q may be NULL; ld_q is not checked).
 *               This is the static min-max calibration of section 3.2: because
 *               fl32(a/448) is monotone in a, the max of the row scales over all
 *               calibration batches equals the scale of the largest magnitude
 *               seen.  The caller sets scales[0] to 0 (or a previous running
 *               value, finite and >= 0) before the first batch; the update is
 *               an atomic max, so the result does not depend on the order of
 *               rows or of calls.
 *
 * E4M3(.) rounds to nearest with ties to the even mantissa and saturates any
 * magnitude above 448 to +-448; NaN gives 0x7F; the sign of zero is kept.
 * fl32(a/b) is the correctly rounded fp32 quotient.  Results are bit-exact
 * given v.  For SILU_MUL, silu(g) = g / (1 + e^-g) is evaluated in fp32 with
 * the hardware exp2 and reciprocal (about 1 ulp each), so bf16(v) can differ
 * from an exact evaluation by one bf16 ulp at near-ties of its rounding.
 *
 * x       bf16 [rows, ld_x]; cols (or 2*cols for SILU_MUL) <= ld_x.
 * scales  fp32 [rows] (PER_ROW, written), fp32 [1] (PER_TENSOR, read; must be
 *         finite and > 0) or fp32 [1] (CALIBRATE, read and updated).
 * q       uint8 [rows, ld_q], cols <= ld_q.
 * Requirements: rows >= 0 (0 is a no-op), cols > 0 and cols % 8 == 0,
 * ld_x % 8 == 0, ld_q % 8 == 0, x and q 16-byte aligned (SPEC_ERR_ALIGN or
 * SPEC_ERR_UNSUPPORTED otherwise).  Non-finite inputs give unspecified codes.
 */
spec_status spec_fp8_quantize(const void* x, int64_t rows, int64_t cols, int64_t ld_x,
                              spec_quant_input in_kind, spec_scale_mode mode,
                              float* scales, uint8_t* q, int64_t ld_q, void* stream);

/*
 * spec_silu_mul_bf16 -- h[r,c] = bf16(silu(x[r,c]) * x[r,cols+c]) without
 * quantizing: exactly the intermediate that SPEC_QIN_SILU_MUL_BF16 quantizes,
 * computed by the same device code.  Same requirements as spec_fp8_quantize;
 * h is bf16 [rows, ld_h], ld_h % 8 == 0, 16-byte aligned.
 */
spec_status spec_silu_mul_bf16(const void* x, int64_t rows, int64_t cols, int64_t ld_x,
                               void* h, int64_t ld_h, void* stream);

/*
 * spec_fp8_clip_count -- how many values a static per-tensor scale clips.
 *
 * The paper judges a static calibration by its activation clip rate: the share
 * of test-time activations outside the per-tensor range set during
 * calibration (section 5, FP8 Calibration Performance).  Read through the
 * quantizer, a value clips when its scaled magnitude leaves the E4M3 range:
 *
 *   count += #{ (r, c) : |fl32(x[r,c] * fl32(1 / scale[0]))| > 448 }
 *
 * which for a scale from SPEC_SCALE_CALIBRATE (s = fl32(amax/448)) is the set
 * of values beyond the calibrated amax, up to the rounding of s and 1/s.  The
 * count is exact (no floating-point summation).
 *
 * x      bf16 [rows, ld_x], cols <= ld_x.
 * scale  fp32 [1], finite and > 0 (read).
 * count  uint64 [1], accumulated: the caller sets it (usually to 0) before the
 *        first call; calls on one counter add up.
 * Requirements: rows >= 0 (0 is a no-op), cols > 0 (SPEC_ERR_SHAPE); cols % 8 == 0
 * (SPEC_ERR_UNSUPPORTED); x 16-byte aligned, ld_x % 8 == 0, scale 4-byte and
 * count 8-byte aligned (SPEC_ERR_ALIGN).
 */
spec_status spec_fp8_clip_count(const void* x, int64_t rows, int64_t cols, int64_t ld_x, const float* scale,
                                uint64_t* count, void* stream);

/*
 * spec_fp8_kv_cache_write -- the verify step's new keys and values, quantized
 * to E4M3 and stored in a paged FP8 KV cache.
 *
 * Section 3.2 (FP8 Post-Training Quantization) stores the KV cache in FP8,
 * half the bytes of bf16.  For every new token t < T whose slot
 * s = slot_mapping[t] lies in [0, num_slots), and every KV head h < H, the
 * key row kx = k[t*ld_k + h*D ...] (D bf16 values) is encoded as
 *
 *   PER_ROW:    sk = max(fl32(max_d |kx[d]| / 448), 2^-100);  k_scale[s*H + h] = sk  (written)
 *   PER_TENSOR: sk = k_scale[0]                                                    (read)
 *   k_cache[(s*H + h)*D + d] = E4M3(fl32(kx[d] * fl32(1 / sk)))
 *
 * and the value rows likewise with v, v_scale and v_cache; the encoding is
 * spec_fp8_quantize's, bit for bit.  A token whose slot is negative (padding)
 * or >= num_slots is skipped: nothing of its rows is written.  Slots of
 * different tokens must differ; if two tokens share a slot, which one's
 * codes (and scales) end up there is unspecified.  The static per-tensor
 * scales of the paper's min-max scheme come from spec_fp8_quantize with
 * SPEC_SCALE_CALIBRATE over calibration keys (or values) viewed as [T, H*D].
 *
 * k, v       bf16 [T, ld_k] / [T, ld_v]; head h of a token at columns [h*D, (h+1)*D);
 *            the K and V column blocks of the QKV projection's output fit directly.
 * slot_mapping  int64 [T].
 * k_scale, v_scale  fp32 [num_slots, H] (PER_ROW, written at the slots stored) or fp32 [1]
 *            (PER_TENSOR, read; finite and > 0).
 * k_cache, v_cache  uint8 [num_slots, H, D] codes: slot-major, so a paged cache of blocks
 *            [num_blocks, block_size, H, D] is the same memory with slot =
 *            block * block_size + offset.  Untouched slots keep their contents.
 * Requirements: T >= 0 (0 is a no-op), H > 0, D > 0, num_slots >= 0, ld_k and ld_v >= H*D
 * (SPEC_ERR_SHAPE); D % 8 == 0 and D <= 512 (SPEC_ERR_UNSUPPORTED); k, v, k_cache and
 * v_cache 16-byte aligned, ld_k and ld_v multiples of 8, slot_mapping 8-byte and the scales
 * 4-byte aligned (SPEC_ERR_ALIGN).  mode must be PER_ROW or PER_TENSOR (SPEC_ERR_ENUM).
 */
spec_status spec_fp8_kv_cache_write(const void* k, int64_t ld_k, const void* v, int64_t ld_v,
                                    const int64_t* slot_mapping, int64_t T, int64_t H, int64_t D,
                                    int64_t num_slots, spec_scale_mode mode, float* k_scale, float* v_scale,
                                    uint8_t* k_cache, uint8_t* v_cache, void* stream);

/*
 * spec_fp8_gemm -- the W8A8 linear layer (section 3.2):
 *
 *   acc[m,n] = sum_k dec(A[m,k]) * dec(W[n,k])     accumulated in fp32
 *   Y[m,n]   = fl32(fl32(acc[m,n] * sa(m)) * sw(n))  then bf16 (RNE) or fp32
 *
 * A       uint8 E4M3 [M, lda] (activations, K contiguous), K <= lda.
 * W       uint8 E4M3 [N, ldw] (weights in nn.Linear layout: row = output channel).
 * a_scale fp32 [M] (PER_ROW) or [1] (PER_TENSOR); w_scale fp32 [N] or [1].
 * Y       bf16 or fp32 [M, ldy], N <= ldy.
 * workspace  device scratch of at least spec_fp8_gemm_workspace_bytes(M,N,K)
 *         bytes (may be NULL when that is 0), 16-byte aligned.  Where the
 *         K dimension is split over workgroups, its first 16 KiB hold one
 *         ticket per output tile: they must be zero before the first call that
 *         uses the workspace (fill it with zeros once, e.g. when allocating),
 *         and every call leaves them zero again, so one workspace serves every
 *         later call of any shape.  The rest of it is overwritten.  Calls that
 *         share a workspace must not overlap (one stream, or serialized).
 * Requirements: M >= 0 (0 is a no-op), N > 0, K > 0, K % 128 == 0 (else
 * SPEC_ERR_UNSUPPORTED); lda % 16 == 0, ldw % 16 == 0, A and W 16-byte
 * aligned; ldy % 8 == 0 and Y 16-byte aligned.  M and N need not be tile
 * multiples.  Products of E4M3 values are exact; only the fp32 accumulation
 * and the epilogue round.
 */
size_t spec_fp8_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K);

spec_status spec_fp8_gemm(const uint8_t* a, int64_t lda, const float* a_scale, spec_scale_mode a_mode,
                          const uint8_t* w, int64_t ldw, const float* w_scale, spec_scale_mode w_mode,
                          int64_t M, int64_t N, int64_t K,
                          void* y, int64_t ldy, spec_out_dtype out_dtype,
                          void* workspace, size_t workspace_bytes, void* stream);

/*
 * spec_fp8_gemm_silu_mul -- the gated FFN's fused gate|up projection with the
 * SiLU gate in its epilogue (the Llama-family target's FFN, section 4), so
 * that the [M, 2I] gate|up output is never written:
 *
 *   yg = bf16_RNE(fl32(fl32(acc[m,c] * sa(m)) * sw(c)))           gate, weight row c
 *   yu = bf16_RNE(fl32(fl32(acc[m,I+c] * sa(m)) * sw(I+c)))       up, weight row I + c
 *   h[m,c] = bf16(silu(yg) * yu)                                  c < I
 *
 * i.e. spec_silu_mul_bf16 applied to spec_fp8_gemm's bf16 output (same device
 * code for the gate), except that K is never split here and the fp32
 * summation order of the accumulators may differ.  h is the input of the
 * down projection's per-token quantize (spec_fp8_quantize, SPEC_QIN_BF16).
 *
 * W       uint8 E4M3 [2I, ldw]: rows 0..I-1 gate, I..2I-1 up (the layout the
 *         SILU_MUL quantize input expects); w_scale [2I] or [1].
 * a, lda, a_scale, a_mode, K: as spec_fp8_gemm.
 * h       bf16 [M, ldh], I <= ldh, ldh % 8 == 0, 16-byte aligned.
 * Requirements: I > 0 (SPEC_ERR_SHAPE), I % 8 == 0 (SPEC_ERR_UNSUPPORTED); the
 * operand requirements of spec_fp8_gemm with N = 2I.  No workspace.
 */
spec_status spec_fp8_gemm_silu_mul(const uint8_t* a, int64_t lda, const float* a_scale, spec_scale_mode a_mode,
                                   const uint8_t* w, int64_t ldw, const float* w_scale, spec_scale_mode w_mode,
                                   int64_t M, int64_t I, int64_t K, void* h, int64_t ldh, void* stream);

/*
 * spec_fp8_gemm_logit_stats -- the LM-head projection of the verify pass (the
 * target model's output layer over the M = B*(k+1) verify rows, hidden size K
 * to vocabulary V; section 3.1) as an FP8 GEMM whose epilogue also produces
 * the acceptance statistics of the logits it writes, so that the acceptance
 * test does not read the target logits a second time for them.
 *
 *   z[m,n] = bf16_RNE(fl32(fl32(acc[m,n] * sa(m)) * sw(n)))   -- spec_fp8_gemm,
 *            bf16 out, except that K is never split here (where spec_fp8_gemm
 *            splits K for this shape the fp32 summation order differs)
 *   for every row m and column group c, 0 <= c < spec_logit_stats_count(M, V, K)
 *   (a group is a contiguous range of columns; the groups, in column order,
 *   partition [0, V); a group may be empty):
 *     temperature > 0:  c2 = fl32(log2(e) / T), t_n = fl32(z[m,n] * c2),
 *                       Mc = max_{n in c} t_n  (= fl32(max z * c2)),
 *                       Zc = sum_{n in c} 2^(t_n - Mc), evaluated in fp32 in an
 *                            unspecified order (partial sums are rescaled as the
 *                            running maximum grows)
 *                       stats[m,c] = (Mc, Zc); an empty group is (-inf, 0)
 *     temperature == 0: stats[m,c] = (max_{n in c} z[m,n], lowest n attaining it as int32 bits);
 *                       an empty group is (-inf, INT32_MAX as int32 bits)
 *   so that max_c Mc and sum_c Zc * 2^(Mc - max) are the row's softmax maximum
 *   and normalizer of z/T in base 2 (the first pass of the acceptance test), and
 *   the best (value, lowest index) pair is the row's argmax (T == 0).
 *
 * a, lda, a_scale, a_mode, w, ldw, w_scale, w_mode, M, K: as spec_fp8_gemm with N = V.
 * logits  bf16 [M, ld_logits]; V <= ld_logits, ld_logits % 8 == 0, 16-byte aligned.
 * stats   pairs of fp32 [M, ld_stats] (ld_stats counted in pairs, >= the group
 *         count), 8-byte aligned.
 * temperature finite and >= 0 (SPEC_ERR_VALUE otherwise).  No workspace.
 * Where the plan takes the 160 x 384 tile (a wide vocabulary), a tile's rows of
 * A and of W must each span at most 4 GiB: 159*lda + 128 <= 2^32 and
 * 383*ldw + 128 <= 2^32 (SPEC_ERR_UNSUPPORTED otherwise).
 * spec_logit_stats_count returns 0 for arguments spec_fp8_gemm would reject.
 */
size_t spec_logit_stats_count(int64_t M, int64_t V, int64_t K);

spec_status spec_fp8_gemm_logit_stats(const uint8_t* a, int64_t lda, const float* a_scale, spec_scale_mode a_mode,
                                      const uint8_t* w, int64_t ldw, const float* w_scale, spec_scale_mode w_mode,
                                      int64_t M, int64_t V, int64_t K, float temperature,
                                      void* logits, int64_t ld_logits, float* stats, int64_t ld_stats,
                                      void* stream);

/*
 * spec_verify_accept -- acceptance of B drafted chains of length k
 * (section 3.1; the rule of the speculative-sampling papers it cites):
 *
 *   temperature == 0 (greedy): g_i = argmax_v target[b,i,v] (lowest index on
 *     ties); keep draft x_i while x_i == g_i; emit g_a at the first mismatch
 *     a, or the bonus g_k after k matches.
 *   temperature > 0 (speculative sampling): p_i = softmax(target[b,i,:]/T),
 *     q_i = softmax(draft[b,i,:]/T) (or one-hot at x_i when draft_logits is
 *     NULL).  For i = 0..k-1: accept x_i iff u[b,i] * q_i(x_i) < p_i(x_i);
 *     at the first rejection emit the smallest v whose cumulative residual
 *     sum_{w<=v} max(0, p_i - q_i)(w) exceeds u[b,k] times the residual's
 *     total, and stop.  If all k are accepted, emit the bonus token drawn the
 *     same way from p_k with u[b,k].
 *
 * target_logits bf16 [B, k+1, V] (position i scores draft i; position k the bonus).
 * draft_logits  bf16 [B, k, V] or NULL.
 * draft_tokens  int32 [B, k]; an id outside [0, V) is a rejection with p = q = 0.
 * uniforms      fp32 [B, k+1] in [0, 1) (ignored when temperature == 0).
 * out_tokens    int32 [B, k+1]: accepted drafts then the emitted token, -1 padded.
 * num_accepted  int32 [B]: a_b in [0, k]; a_b + 1 tokens are emitted.
 * workspace     >= spec_verify_accept_workspace_bytes(B, k, V) bytes; contents on
 *               entry are ignored.
 * Requirements: B >= 0 (0 is a no-op), 1 <= k <= 16, 1 <= V <= 2^22 and
 * B*(2k+1) <= 65535 (SPEC_ERR_UNSUPPORTED otherwise);
 * temperature finite and >= 0 (SPEC_ERR_VALUE otherwise).  Probabilities are
 * computed in fp32; a decision within ~1e-5 relative of its boundary may
 * differ from an exact evaluation.
 */
size_t spec_verify_accept_workspace_bytes(int64_t B, int64_t k, int64_t V);

spec_status spec_verify_accept(const void* target_logits, const void* draft_logits,
                               const int32_t* draft_tokens, const float* uniforms,
                               int64_t B, int64_t k, int64_t V, float temperature,
                               int32_t* out_tokens, int32_t* num_accepted,
                               void* workspace, size_t workspace_bytes, void* stream);

/*
 * spec_verify_accept_noalloc -- spec_verify_accept for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): no workspace argument.  The kernels use
 * a fixed scratch buffer that the library holds in device memory instead, of
 * SPEC_ACCEPT_SCRATCH_BYTES (16 MiB) per GPU, held until the process ends.
 * The scratch is that of the current device (hipGetDevice), which must be
 * the device of `stream`; its address is looked up on the first call on each
 * device.  Nothing is allocated or freed, here or in any later call.
 *
 * Arguments, requirements and results are those of spec_verify_accept.  A
 * call whose spec_verify_accept_workspace_bytes(B, k, V) exceeds
 * SPEC_ACCEPT_SCRATCH_BYTES returns SPEC_ERR_SCRATCH before any HIP call
 * (at k = 4, V = 128256 that allows B up to about 850).  Every call on one
 * GPU shares that GPU's scratch and leaves it holding its own intermediate
 * values (no call depends on what is there on entry), so calls that overlap
 * on one GPU -- on different streams, or from different threads -- race and
 * must be serialized by the caller.
 */
#define SPEC_ACCEPT_SCRATCH_BYTES ((size_t)16 << 20)

spec_status spec_verify_accept_noalloc(const void* target_logits, const void* draft_logits,
                                       const int32_t* draft_tokens, const float* uniforms,
                                       int64_t B, int64_t k, int64_t V, float temperature,
                                       int32_t* out_tokens, int32_t* num_accepted, void* stream);

/*
 * spec_verify_accept_stats -- spec_verify_accept with the target rows'
 * statistics taken from spec_fp8_gemm_logit_stats (called with the same
 * temperature on the rows of target_logits) instead of computed from
 * target_logits: only draft_logits, when given, are streamed for theirs, and
 * target_logits are read only at the draft tokens and in the row of the
 * sampled position.
 *
 * target_stats  pairs of fp32 [B*(k+1), ld_stats], row i*(k+1)+p for sequence i,
 *               position p (the row order of target_logits); n_stats entries per row,
 *               1 <= n_stats <= ld_stats, n_stats < 2^31; 8-byte aligned.
 * All other arguments, requirements, workspace and results as spec_verify_accept.
 * The results equal spec_verify_accept's except for a decision within the fp32
 * rounding of the statistics of its boundary (their summation order differs).
 */
spec_status spec_verify_accept_stats(const void* target_logits, const float* target_stats,
                                     int64_t n_stats, int64_t ld_stats, const void* draft_logits,
                                     const int32_t* draft_tokens, const float* uniforms,
                                     int64_t B, int64_t k, int64_t V, float temperature,
                                     int32_t* out_tokens, int32_t* num_accepted,
                                     void* workspace, size_t workspace_bytes, void* stream);

/*
 * spec_verify_accept_tree -- acceptance of B drafted token TREES, the
 * standard EAGLE drafting mode the paper compares with greedy chains (the
 * appendix's tree versus greedy drafting; Table 2's tree rows).  The target
 * scored every node in one pass (tree attention, outside this library).
 *
 * Tree of sequence b: N nodes; parents[b,n] in [-1, n) is node n's parent (-1:
 * a candidate for the first new token); tokens[b,n] its drafted token.  The
 * children of a node are its candidates, in index order.  Target row 0 scores
 * the first new position, row n+1 the position after node n.
 *
 *   temperature == 0: from the root, move to the first child whose token is
 *     the argmax of the current row (lowest index on ties); where none
 *     matches, emit that argmax.
 *   temperature > 0: the candidates are deterministic proposals (one-hot
 *     draft distributions, e.g. a top-k expansion).  With P = softmax(row/T)
 *     at the current node, child n (token x) is accepted iff
 *     u[b,n] * (1 - S) < P(x), S the mass of the tokens already rejected at
 *     this node (a repeated token has P = 0); on acceptance the walk moves to
 *     n, else x is removed.  Where every child is rejected (or there is none),
 *     emit the smallest v whose cumulative sum of P without the removed
 *     tokens exceeds u[b,N] times that residual's total (P itself if the
 *     residual vanished).  This is sequential sampling from P: the emitted
 *     tokens follow the target distribution exactly.  With parents = [-1, 0,
 *     .., N-2] it is spec_verify_accept with draft_logits NULL and k = N.
 *
 * target_logits  bf16 [B, N+1, V].
 * parents, tokens int32 [B, N]; a node whose parent is outside [-1, n) is never
 *                accepted; a token outside [0, V) is a rejection with P = 0.
 * uniforms       fp32 [B, N+1] in [0, 1): u[b,n] tests node n, u[b,N] is the final
 *                draw (ignored when temperature == 0).
 * out_tokens     int32 [B, N+1]: the accepted path's tokens, then the emitted token,
 *                -1 padded.
 * accepted_nodes int32 [B, N]: the accepted path's node indices, -1 padded.
 * num_accepted   int32 [B]: path length a_b; a_b + 1 tokens are emitted.
 * workspace      >= spec_verify_accept_tree_workspace_bytes(B, N, V); contents on entry
 *                are ignored.
 * Requirements: B >= 0 (0 is a no-op), 1 <= N <= 64, 1 <= V <= 2^22, B <= 65535,
 * B*(N+1)*ceil(V/4096) < 2^31 (SPEC_ERR_UNSUPPORTED otherwise); temperature finite
 * and >= 0 (SPEC_ERR_VALUE).
 * Probabilities are computed in fp32 (the accept tests in double from fp32
 * statistics); a decision within ~1e-5 relative of its boundary may differ from
 * an exact evaluation.
 */
size_t spec_verify_accept_tree_workspace_bytes(int64_t B, int64_t N, int64_t V);

spec_status spec_verify_accept_tree(const void* target_logits, const int32_t* parents, const int32_t* tokens,
                                    const float* uniforms, int64_t B, int64_t N, int64_t V, float temperature,
                                    int32_t* out_tokens, int32_t* accepted_nodes, int32_t* num_accepted,
                                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * spec_tree_attention_mask -- the attention mask of B drafted trees for the
 * target's single scoring pass over every node (tree attention, the EAGLE
 * tree mode of the appendix's tree versus greedy drafting).
 *
 * The row of node n may attend to the prefix, the root (the last accepted
 * token) and exactly the tree nodes on the path from the root to n, n
 * included; a node of another branch is another continuation and stays
 * hidden.  For every node:
 *
 *   mask[b,n]  bit j (j < N) set iff node j lies on that path;
 *   depth[b,n] the number of nodes on it (the node sits depth[b,n] positions
 *              after the root, which gives its position id).
 *
 * A node whose chain of parents leaves [-1, m) at some node m (the encoding
 * of spec_verify_accept_tree) is unreachable: mask 0 and depth 0, and so is
 * every node below it.  For an accepted path (accepted_nodes of
 * spec_verify_accept_tree), the mask of its last node holds exactly the path.
 *
 * parents  int32 [B, N] as for spec_verify_accept_tree.
 * mask     uint64 [B, N] (8-byte aligned); depth int32 [B, N].
 * Requirements: B >= 0 (0 is a no-op), N >= 1 (SPEC_ERR_SHAPE); N <= 64 and
 * ceil(B/4) < 2^31 (SPEC_ERR_UNSUPPORTED).
 */
spec_status spec_tree_attention_mask(const int32_t* parents, int64_t B, int64_t N, uint64_t* mask, int32_t* depth,
                                     void* stream);

/* Static description of a status code (never NULL). */
const char* spec_status_string(spec_status s);

/* hipError_t value of the last SPEC_ERR_HIP returned on this thread (0 if none). */
int spec_last_hip_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int spec_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SPEC_FP8_H */
