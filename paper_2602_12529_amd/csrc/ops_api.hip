// C ABI of the kernel-level building blocks (include/ff_ops.h): validation + dispatch.
#include <climits>
#include <cmath>

#include "../../include/ff_ops.h"
#include "ff_internal.h"

using namespace ff;

namespace {
int check_dtype(const char* fn, int32_t dt) {
  if (dt != FF_F32 && dt != FF_BF16) return fail(FF_EINVAL, "%s: bad dtype %d", fn, dt);
  return FF_OK;
}

// Size limits of the linear layers and attention: row strides and K fit the 32-bit offsets of a
// tile's buffer loads, and tile and workgroup counts fit a launch grid.
constexpr int64_t kMaxOpRows = int64_t(1) << 27, kMaxOpStride = int64_t(1) << 22;
int check_linear_sizes(const char* fn, int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldw, int64_t ldo,
                       int64_t ldr, int64_t gate_ld) {
  if (M > kMaxOpRows || N > kMaxOpRows || K > kMaxOpStride || lda > kMaxOpStride || ldw > kMaxOpStride ||
      ldo > kMaxOpStride || ldr > kMaxOpStride || gate_ld > kMaxOpStride || ((M + 127) / 128) * ((N + 127) / 128) > INT32_MAX)
    return fail(FF_EUNSUPPORTED, "%s: M, N above 2^27, K or a row stride above 2^22, or too many tiles", fn);
  return FF_OK;
}
}  // namespace

extern "C" {

int ff_linear(const void* A, int64_t lda, const void* W, const void* bias, void* out, int64_t ldo, int64_t M,
              int64_t N, int64_t K, int32_t epi, int64_t gelu_from, const float* gate, int64_t gate_ld,
              const void* resid, int64_t ldr, int64_t rows_per_sample, int32_t dtype, void* workspace,
              size_t ws_bytes, void* stream) {
  const char* fn = "ff_linear";
  FF_TRY(check_dtype(fn, dtype));
  if (M < 0 || N < 0 || K < 1) return fail(FF_EINVAL, "%s: bad shape M=%lld N=%lld K=%lld", fn, (long long)M, (long long)N, (long long)K);
  if (M == 0 || N == 0) return FF_OK;
  if (!A || !W || !out) return fail(FF_EINVAL, "%s: null A, W or out", fn);
  if (lda < K || ldo < N) return fail(FF_EINVAL, "%s: lda < K or ldo < N", fn);
  FF_TRY(check_linear_sizes(fn, M, N, K, lda, K, ldo, epi == FF_EPI_GATED ? ldr : 0, gate ? gate_ld : 0));
  if (epi < FF_EPI_BIAS || epi > FF_EPI_GATED) return fail(FF_EINVAL, "%s: bad epilogue %d", fn, epi);
  if (epi == FF_EPI_GATED) {
    if (!resid) return fail(FF_EINVAL, "%s: gated epilogue needs resid", fn);
    if (ldr < N || (gate && (rows_per_sample < 1 || gate_ld < N))) return fail(FF_EINVAL, "%s: bad gate/resid layout", fn);
  }
  if (!aligned16(A) || !aligned16(W) || !aligned16(out)) return fail(FF_EINVAL, "%s: pointers must be 16-byte aligned", fn);
  if (dtype == FF_BF16) {
    if (K % 64) return fail(FF_EUNSUPPORTED, "%s: bf16 needs K %% 64 == 0 (K=%lld)", fn, (long long)K);
    if (lda % 8) return fail(FF_EINVAL, "%s: bf16 needs lda %% 8 == 0", fn);
  }
  GemmArgs g{};
  g.dtype = dtype;
  g.M = M; g.N = N; g.K = K;
  g.A1 = A; g.lda1 = lda; g.K1 = K; g.A2 = nullptr; g.lda2 = 0;
  g.W = W; g.ldw = K; g.bias = bias;
  g.out = out; g.ldo = ldo;
  g.epi = epi; g.gelu_from = gelu_from;
  g.gate = gate; g.gate_ld = gate_ld; g.resid = resid; g.ldr = ldr;
  g.rows_per_sample = rows_per_sample > 0 ? rows_per_sample : M;
  if (workspace) {
    if (!aligned16(workspace)) return fail(FF_EINVAL, "%s: workspace must be 16-byte aligned", fn);
    g.split_ws = workspace;
    g.split_bytes = ws_bytes;
  }
  return gemm(g, static_cast<hipStream_t>(stream));
}

int ff_linear_workspace_size(size_t* bytes) {
  if (!bytes) return fail(FF_EINVAL, "ff_linear_workspace_size: null output");
  *bytes = gemm_split_bytes();
  return FF_OK;
}

int ff_attention(const void* Q, const void* K, const void* V, void* out, int64_t B, int64_t heads, int64_t n_q,
                 int64_t n_kv, int64_t head_dim, int32_t dtype, void* stream) {
  const char* fn = "ff_attention";
  FF_TRY(check_dtype(fn, dtype));
  if (B < 0 || heads < 1 || n_q < 0 || n_kv < 1 || head_dim < 1) return fail(FF_EINVAL, "%s: bad shape", fn);
  if (B == 0 || n_q == 0) return FF_OK;
  if (!Q || !K || !V || !out) return fail(FF_EINVAL, "%s: null pointer", fn);
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(out)) return fail(FF_EINVAL, "%s: pointers must be 16-byte aligned", fn);
  if (B > kMaxOpRows || heads > kMaxOpStride || n_q > kMaxOpRows || n_kv > kMaxOpRows || heads * head_dim > kMaxOpStride ||
      (n_q + 63) / 64 * B * heads > INT32_MAX)
    return fail(FF_EUNSUPPORTED, "%s: n_q or n_kv above 2^27, heads x head_dim above 2^22, or too many workgroups", fn);
  AttnArgs a{};
  a.dtype = dtype;
  a.B = B; a.heads = heads; a.d = head_dim; a.n_q = n_q; a.n_kv = n_kv;
  a.Q = Q; a.K = K; a.Vt = V;
  a.out0 = out; a.out1 = out; a.split = n_q; a.ldo = heads * head_dim;
  a.scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(head_dim)));
  return attention(a, static_cast<hipStream_t>(stream));
}

int ff_norm_modulate(const void* x, void* y, int64_t rows, int64_t H, const float* shift, const float* scale,
                     int64_t mod_ld, int64_t rows_per_sample, int32_t norm_kind, float eps, int32_t dtype,
                     void* stream) {
  const char* fn = "ff_norm_modulate";
  FF_TRY(check_dtype(fn, dtype));
  if (rows < 0 || H < 1) return fail(FF_EINVAL, "%s: bad shape", fn);
  if (rows == 0) return FF_OK;
  if (rows > kMaxOpRows || H > kMaxOpStride || mod_ld > kMaxOpStride)
    return fail(FF_EUNSUPPORTED, "%s: rows above 2^27, or H or mod_ld above 2^22", fn);
  if (!x || !y) return fail(FF_EINVAL, "%s: null x or y", fn);
  if (norm_kind != FF_NORM_RMS && norm_kind != FF_NORM_LN) return fail(FF_EINVAL, "%s: bad norm_kind", fn);
  if (!(eps > 0.f)) return fail(FF_EINVAL, "%s: eps must be > 0", fn);
  if ((shift || scale) && (rows_per_sample < 1 || mod_ld < H)) return fail(FF_EINVAL, "%s: bad modulation layout", fn);
  NormArgs a{};
  a.dtype = dtype;
  a.rows = rows; a.H = H;
  a.x = x; a.ldx = H; a.y = y; a.ldy = H;
  a.norm_kind = norm_kind; a.eps = eps;
  a.shift = shift; a.scale = scale; a.mod_ld = mod_ld;
  a.w = nullptr; a.bias = nullptr;
  a.rows_per_sample = rows_per_sample > 0 ? rows_per_sample : rows;
  return norm_modulate(a, static_cast<hipStream_t>(stream));
}

int ff_qk_norm_rope(const void* qkv, int64_t B, int64_t n_tok, int64_t heads, int64_t head_dim, const void* q_w,
                    const void* k_w, float eps, const float* rope, void* Q, void* K, void* V, int64_t n_joint,
                    int64_t tok_offset, int32_t dtype, void* stream) {
  const char* fn = "ff_qk_norm_rope";
  FF_TRY(check_dtype(fn, dtype));
  if (B < 0 || n_tok < 0 || heads < 1 || head_dim < 2 || head_dim % 2 || head_dim > 128)
    return fail(FF_EINVAL, "%s: bad shape", fn);
  if (tok_offset < 0 || tok_offset + n_tok > n_joint) return fail(FF_EINVAL, "%s: tokens outside the joint sequence", fn);
  if (B == 0 || n_tok == 0) return FF_OK;
  if (B > 65535 || heads > 65535 || n_joint > kMaxOpRows || heads * head_dim > kMaxOpStride)
    return fail(FF_EUNSUPPORTED, "%s: B or heads above 65535, n_joint above 2^27 or heads x head_dim above 2^22", fn);
  if (!qkv || !q_w || !k_w || !Q || !K || !V) return fail(FF_EINVAL, "%s: null pointer", fn);
  QkvArgs a{};
  a.dtype = dtype;
  a.B = B; a.n_tok = n_tok; a.tok_offset = tok_offset; a.n_joint = n_joint; a.src_rows = n_tok;
  a.heads = static_cast<int>(heads); a.d = static_cast<int>(head_dim);
  const size_t es = dtype_size(dtype), H = static_cast<size_t>(heads * head_dim);
  a.q = qkv; a.k = static_cast<const char*>(qkv) + H * es; a.v = static_cast<const char*>(qkv) + 2 * H * es;
  a.ld = static_cast<int64_t>(3 * H);
  a.q_w = q_w; a.k_w = k_w; a.full_width_norm = 0; a.apply_norm = 1; a.eps = eps;
  a.rope = reinterpret_cast<const float2*>(rope);
  a.Q = Q; a.Kd = K; a.Vt = V;
  a.v_transposed = dtype == FF_BF16;
  return qk_norm_rope(a, static_cast<hipStream_t>(stream));
}

int ff_rope_table(float* out, const int32_t grid[3], int32_t head_dim, const int32_t axes[3], double theta,
                  void* stream) {
  const char* fn = "ff_rope_table";
  if (!out || !grid || !axes) return fail(FF_EINVAL, "%s: null pointer", fn);
  if (grid[0] < 1 || grid[1] < 1 || grid[2] < 1) return fail(FF_EINVAL, "%s: bad grid", fn);
  const int64_t n01 = static_cast<int64_t>(grid[0]) * grid[1];   // both factors < 2^31: no overflow
  if (n01 > kMaxOpRows || n01 * grid[2] > kMaxOpRows || head_dim > 1024)
    return fail(FF_EUNSUPPORTED, "%s: more than 2^27 grid positions or head_dim above 1024", fn);
  if (head_dim < 2 || head_dim % 2 || axes[0] % 2 || axes[1] % 2 || axes[2] % 2 || axes[0] < 0 || axes[1] < 0 ||
      axes[2] < 0 || static_cast<int64_t>(axes[0]) + axes[1] + axes[2] != head_dim)
    return fail(FF_EINVAL, "%s: axes must be even and sum to head_dim", fn);
  if (!(theta > 0)) return fail(FF_EINVAL, "%s: theta must be > 0", fn);
  return rope_table(reinterpret_cast<float2*>(out), grid, head_dim, axes, theta, static_cast<hipStream_t>(stream));
}

int ff_skinny_linear(const float* in, const void* W, const void* bias, float* out, int64_t B, int64_t N, int64_t K,
                     int32_t act_in, int32_t act_out, int32_t dtype, const int32_t* classes, void* stream) {
  const char* fn = "ff_skinny_linear";
  FF_TRY(check_dtype(fn, dtype));
  if (B < 0 || N < 0 || K < 1) return fail(FF_EINVAL, "%s: bad shape", fn);
  if (B == 0 || N == 0) return FF_OK;
  if (!in || !W || !out) return fail(FF_EINVAL, "%s: null pointer", fn);
  if (K % 8) return fail(FF_EUNSUPPORTED, "%s: K must be a multiple of 8", fn);
  if (B > 65535 || N > kMaxOpRows || K > kMaxOpStride)
    return fail(FF_EUNSUPPORTED, "%s: B above 65535, N above 2^27 or K above 2^22", fn);
  if (act_in < 0 || act_in > 2 || act_out < 0 || act_out > 2) return fail(FF_EINVAL, "%s: bad activation", fn);
  if (!aligned16(in) || !aligned16(W)) return fail(FF_EINVAL, "%s: pointers must be 16-byte aligned", fn);
  SkinnyArgs a{};
  a.dtype = dtype;
  a.B = B; a.N = N; a.K = K;
  a.in = in; a.ldi = K; a.act_in = act_in;
  a.W = W; a.bias = bias;
  a.out = out; a.ldo = N;
  a.accumulate = 0; a.act_out = act_out;
  a.rowmap = classes;
  return skinny_linear(a, static_cast<hipStream_t>(stream));
}

int ff_row_classes(const float* c, int64_t B, int64_t H, int32_t* map, void* stream) {
  const char* fn = "ff_row_classes";
  if (B < 0 || H < 1) return fail(FF_EINVAL, "%s: bad shape B=%lld H=%lld", fn, (long long)B, (long long)H);
  if (B == 0) return FF_OK;
  if (!c || !map) return fail(FF_EINVAL, "%s: null pointer", fn);
  return row_classes(c, B, H, map, static_cast<hipStream_t>(stream));
}

int ff_quantize_fp8(const void* x, int64_t ldx, uint8_t* q, int64_t ldq, float* d, int64_t rows, int64_t cols,
                    int32_t dtype, void* stream) {
  const char* fn = "ff_quantize_fp8";
  FF_TRY(check_dtype(fn, dtype));
  if (rows < 0 || cols < 0) return fail(FF_EINVAL, "%s: bad shape rows=%lld cols=%lld", fn, (long long)rows, (long long)cols);
  if (rows == 0) return FF_OK;
  if (!x || !q || !d) return fail(FF_EINVAL, "%s: null x, q or d", fn);
  if (ldx < cols || ldq < cols) return fail(FF_EINVAL, "%s: ldx or ldq < cols", fn);
  if (cols % 8 || ldx % 8 || ldq % 8) return fail(FF_EUNSUPPORTED, "%s: cols, ldx and ldq must be multiples of 8", fn);
  if (rows > kMaxOpRows || ldx > kMaxOpStride || ldq > kMaxOpStride)
    return fail(FF_EUNSUPPORTED, "%s: rows above 2^27 or a row stride above 2^22", fn);
  if (!aligned16(x) || !aligned16(q)) return fail(FF_EINVAL, "%s: x and q must be 16-byte aligned", fn);
  return quantize_fp8(dtype, x, ldx, q, ldq, d, rows, cols, static_cast<hipStream_t>(stream));
}

int ff_linear_fp8(const uint8_t* A, int64_t lda, const float* d_a, const uint8_t* W, int64_t ldw, const float* d_w,
                  const void* bias, void* out, int64_t ldo, int64_t M, int64_t N, int64_t K, int32_t epi,
                  int64_t gelu_from, void* stream) {
  const char* fn = "ff_linear_fp8";
  if (M < 0 || N < 0 || K < 1) return fail(FF_EINVAL, "%s: bad shape M=%lld N=%lld K=%lld", fn, (long long)M, (long long)N, (long long)K);
  if (M == 0 || N == 0) return FF_OK;
  if (!A || !W || !d_a || !d_w || !out) return fail(FF_EINVAL, "%s: null A, W, d_a, d_w or out", fn);
  if (lda < K || ldw < K || ldo < N) return fail(FF_EINVAL, "%s: lda or ldw < K, or ldo < N", fn);
  FF_TRY(check_linear_sizes(fn, M, N, K, lda, ldw, ldo, 0, 0));
  if (epi != FF_EPI_BIAS && epi != FF_EPI_GELU) return fail(FF_EINVAL, "%s: epilogue %d (bias or GELU only)", fn, epi);
  if (K % 128) return fail(FF_EUNSUPPORTED, "%s: K %% 128 != 0 (K=%lld)", fn, (long long)K);
  if (lda % 16 || ldw % 16 || ldo % 8) return fail(FF_EINVAL, "%s: lda, ldw %% 16 and ldo %% 8 must be 0", fn);
  if (!aligned16(A) || !aligned16(W) || !aligned16(out) || !aligned16(d_w) || (bias && !aligned16(bias)))
    return fail(FF_EINVAL, "%s: A, W, out, bias and d_w must be 16-byte aligned", fn);
  Fp8GemmArgs g{};
  g.M = M; g.N = N; g.K = K;
  g.A = A; g.lda = lda; g.d_a = d_a;
  g.W = W; g.ldw = ldw; g.d_w = d_w;
  g.bias = bias; g.out = out; g.ldo = ldo;
  g.epi = epi == FF_EPI_GELU ? EPI_GELU : EPI_NONE;
  g.gelu_from = gelu_from;
  return gemm_fp8(g, static_cast<hipStream_t>(stream));
}

int ff_stream_probe(int32_t mode, int32_t nontemporal, const void* src, void* dst, int64_t bytes, int32_t blocks,
                    void* stream) {
  const char* fn = "ff_stream_probe";
  if (mode < 0 || mode > 2) return fail(FF_EINVAL, "%s: mode %d (0 read, 1 write, 2 copy)", fn, mode);
  if (bytes < 0 || bytes % 16) return fail(FF_EINVAL, "%s: bytes=%lld must be a non-negative multiple of 16", fn, (long long)bytes);
  if (blocks < 1 || blocks > (1 << 20)) return fail(FF_EINVAL, "%s: blocks=%d outside [1, 2^20]", fn, blocks);
  if (bytes == 0) return FF_OK;
  if ((mode != 1 && !src) || !dst) return fail(FF_EINVAL, "%s: null buffer", fn);
  if ((src && !aligned16(src)) || !aligned16(dst)) return fail(FF_EINVAL, "%s: buffers must be 16-byte aligned", fn);
  return stream_probe(mode, nontemporal != 0, src, dst, bytes / 16, blocks, static_cast<hipStream_t>(stream));
}

}  // extern "C"
