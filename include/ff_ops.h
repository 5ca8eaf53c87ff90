/*
 * ff_ops.h -- kernel-level entry points of libff.so.
 *
 * These expose the building blocks that ff_dit_forward composes, so each can
 * be checked and timed on its own at full shape.  Conventions (ownership,
 * asynchrony on `stream`, host-side validation, status codes, ff_last_error)
 * are those of ff.h.  All tensors are device memory, row-major, of `dtype`
 * (FF_F32 or FF_BF16) unless stated otherwise.
 */
#ifndef FF_OPS_H
#define FF_OPS_H

#include "ff.h"

#ifdef __cplusplus
extern "C" {
#endif

enum { FF_EPI_BIAS = 0, FF_EPI_GELU = 1, FF_EPI_GATED = 2 };

/* Linear layer out = epi(A W^T + bias) of the DiT blocks.
 *   A [M, K] (row stride lda), W [N, K] (nn.Linear layout, row stride K),
 *   bias [N] or NULL, out [M, N] (row stride ldo).
 *   FF_EPI_BIAS:  out = A W^T + bias
 *   FF_EPI_GELU:  out = GELU_tanh(A W^T + bias) on columns >= gelu_from
 *                 (earlier columns get A W^T + bias)
 *   FF_EPI_GATED: out = resid + gate[m / rows_per_sample] * (A W^T + bias), the
 *                 adaLN-gated residual; gate float32 [*, gate_ld] or NULL for a
 *                 plain residual (gate = 1), resid [M, N] (row stride ldr) may
 *                 alias out.
 * Accumulation is float32.  bf16 requires K % 64 == 0 and lda, ldo, ldr % 8 == 0.  Limits
 * (FF_EUNSUPPORTED): M, N <= 2^27; K and the row strides <= 2^22 elements; at most 2^31 - 1
 * tiles of 128 x 128.
 * workspace (device, 16-byte aligned, ff_linear_workspace_size bytes) or NULL: with it, a bf16
 * launch whose 256 x 256 tiles leave a last, partly filled round of the GPU's compute units splits
 * that round's tiles along K (float32 partial sums in the workspace, added in a fixed order, so the
 * result is deterministic); without it nothing is split.  The workspace holds nothing between
 * calls; calls that overlap on one workspace race. */
int ff_linear(const void* A, int64_t lda, const void* W, const void* bias, void* out, int64_t ldo,
              int64_t M, int64_t N, int64_t K, int32_t epi, int64_t gelu_from, const float* gate,
              int64_t gate_ld, const void* resid, int64_t ldr, int64_t rows_per_sample, int32_t dtype,
              void* workspace, size_t ws_bytes, void* stream);

/* Workspace bytes of ff_linear's split-K tail (the same for every shape). */
int ff_linear_workspace_size(size_t* bytes);

/* Attention O = softmax(Q K^T / sqrt(d)) V, no mask.
 *   Q [B, heads, n_q, d], K [B, heads, n_kv, d];
 *   V: bf16 takes V transposed, [B, heads, d, n_kv]; f32 takes [B, heads, n_kv, d].
 *   out [B, n_q, heads*d] (token-major, heads concatenated).
 * bf16: d == 128, n_kv % 8 == 0.  f32: d <= 64, B heads <= 65535.  Limits (FF_EUNSUPPORTED):
 * n_q, n_kv <= 2^27, heads d <= 2^22, at most 2^31 - 1 workgroups of 64 queries. */
int ff_attention(const void* Q, const void* K, const void* V, void* out, int64_t B, int64_t heads,
                 int64_t n_q, int64_t n_kv, int64_t head_dim, int32_t dtype, void* stream);

/* y = Norm(x) (1 + scale[b]) + shift[b] per row, b = row / rows_per_sample.
 * x, y [rows, H]; shift, scale float32 rows of stride mod_ld (either may be NULL);
 * norm_kind FF_NORM_RMS or FF_NORM_LN (no affine), statistics in float32.  rows <= 2^27, H and
 * mod_ld <= 2^22 (FF_EUNSUPPORTED). */
int ff_norm_modulate(const void* x, void* y, int64_t rows, int64_t H, const float* shift,
                     const float* scale, int64_t mod_ld, int64_t rows_per_sample, int32_t norm_kind,
                     float eps, int32_t dtype, void* stream);

/* Per-head RMSNorm (weights q_w, k_w of [d]) and RoPE of one token stream, with
 * relayout into the joint attention layout.
 *   qkv [B, n_tok, 3*heads*d] (Q | K | V per row);
 *   rope: float32 pairs [n_tok, d/2, 2] = (cos, sin), or NULL for no rotation;
 *   Q, K out [B, heads, n_joint, d] at token offset tok_offset;
 *   V out transposed [B, heads, d, n_joint] (bf16) or [B, heads, n_joint, d] (f32).
 * B, heads <= 65535, n_joint <= 2^27, heads d <= 2^22 (FF_EUNSUPPORTED). */
int ff_qk_norm_rope(const void* qkv, int64_t B, int64_t n_tok, int64_t heads, int64_t head_dim,
                    const void* q_w, const void* k_w, float eps, const float* rope, void* Q, void* K,
                    void* V, int64_t n_joint, int64_t tok_offset, int32_t dtype, void* stream);

/* RoPE (cos, sin) table for a (frames, rows, cols) grid: out float32 [N, d/2, 2],
 * pair i of band a turning by pos_a * theta^(-2i/axes[a]) (float64 math).  At most 2^27 grid
 * positions and head_dim <= 1024 (FF_EUNSUPPORTED). */
int ff_rope_table(float* out, const int32_t grid[3], int32_t head_dim, const int32_t axes[3],
                  double theta, void* stream);

/* out[b, n] = act_out(sum_k W[n,k] act_in(in[b,k]) + bias[n]) for skinny batches
 * (the adaLN modulation and embedding MLPs).  in float32 [B, K], out float32
 * [B, N], W of dtype [N, K]; act: 0 none, 1 SiLU, 2 GELU_tanh.  classes: NULL, or the row map
 * ff_row_classes made of `in` (device): then each class is computed once and its result stored
 * in every member's row (the same values, since members are bitwise-equal rows).  K % 8 == 0;
 * limits (FF_EUNSUPPORTED): B <= 65535, N <= 2^27, K <= 2^22. */
int ff_skinny_linear(const float* in, const void* W, const void* bias, float* out, int64_t B, int64_t N,
                     int64_t K, int32_t act_in, int32_t act_out, int32_t dtype, const int32_t* classes,
                     void* stream);

/* Classes of bitwise-equal rows of c (float32 [B, H], device, 16-byte aligned, H % 4 == 0): in a
 * rollout step every sample of a prompt has the same conditioning c = f(t, prompt) (Eq. 1's
 * v_theta(x_t, c, t)), so ff_dit_forward computes each adaLN modulation vector once per class.
 * map (int32 device, 2 + 3 B entries): map[0] = U, the number of classes; map[1 + j], j < U, the
 * first row of class j (ascending); map[1 + B + j], j <= U, the start of class j in the member
 * list; map[2 + 2 B + m], m < B, the members grouped by class, ascending within a class.  For
 * B > 64 every row is its own class.  Errors: FF_EINVAL (null pointers, B < 0, H < 1),
 * FF_EUNSUPPORTED (H % 4, misaligned c). */
int ff_row_classes(const float* c, int64_t B, int64_t H, int32_t* map, void* stream);

/* HBM streaming probe (measurement, not part of the method): mode 0 reads `bytes` from src (each
 * workgroup folds what it read into one 16-byte word of dst, which must hold `blocks` of them),
 * mode 1 writes `bytes` to dst, mode 2 copies src to dst; 16-byte accesses, four in flight per
 * thread, `blocks` workgroups of 256 threads in a grid-stride loop, non-temporal loads and stores
 * when `nontemporal` is set.  It gives the achievable streaming bandwidth that the HBM-bound
 * kernels are compared with.  bytes % 16 == 0; buffers 16-byte aligned. */
int ff_stream_probe(int32_t mode, int32_t nontemporal, const void* src, void* dst, int64_t bytes, int32_t blocks,
                    void* stream);

/* FP8 row quantisation to OCP E4M3 (sign, 4 exponent bits with bias 7, 3 mantissa bits; largest
 * magnitude 448, no infinities).  Not from the paper, whose DiT runs its linear layers in bf16:
 * the FP8 layer below is a throughput variant of ff_linear.
 * For each row r of x [rows, cols] (dtype, row stride ldx elements): amax = max |x[r, :]|,
 * q[r, :] = round-to-nearest-even(x[r, :] * fl32(448 / amax)) as codes (uint8, row stride ldq
 * bytes; a value that rounds to zero keeps its sign bit) and d[r] = fl32(amax / 448) (float32), so
 * that x[r, k] ~ d[r] * decode(q[r, k]).  A row with amax < 448 * 2^-126 (a row of zeros
 * included) gets codes 0 and d = 0; a row holding an infinity or a NaN gets the NaN code 0x7f in
 * every position and d = NaN.  cols, ldx, ldq % 8 == 0; x and q 16-byte aligned; rows <= 2^27 and
 * ldx, ldq <= 2^22 (FF_EUNSUPPORTED). */
int ff_quantize_fp8(const void* x, int64_t ldx, uint8_t* q, int64_t ldq, float* d, int64_t rows, int64_t cols,
                    int32_t dtype, void* stream);

/* FP8 linear layer out = epi(d_a[m] * d_w[n] * (A W^T)[m, n] + bias[n]): A [M, K] and W [N, K]
 * E4M3 codes (row strides lda, ldw in bytes), d_a [M] and d_w [N] their float32 scales (as
 * ff_quantize_fp8 produces them), bias bf16 [N] or NULL, out bf16 [M, N] (row stride ldo
 * elements); epi FF_EPI_BIAS or FF_EPI_GELU (GELU_tanh on columns >= gelu_from).  Products of
 * codes accumulate in float32.  K % 128 == 0; lda, ldw % 16 == 0; ldo % 8 == 0; A, W, out,
 * bias and d_w 16-byte aligned.  Size limits as ff_linear. */
int ff_linear_fp8(const uint8_t* A, int64_t lda, const float* d_a, const uint8_t* W, int64_t ldw, const float* d_w,
                  const void* bias, void* out, int64_t ldo, int64_t M, int64_t N, int64_t K, int32_t epi,
                  int64_t gelu_from, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* FF_OPS_H */
