// Internal declarations shared by the library's translation units (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>

#include <atomic>
#include <cstdint>
#include <cstdio>
#include <string>

#include "../../include/ff.h"

namespace ff {

// ----------------------------------------------------------------- errors
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int hip_status(hipError_t e, const char* what);   // FF_OK or FF_EHIP with message

#define FF_CHECK_HIP(expr, what)                             \
  do {                                                       \
    hipError_t _e = (expr);                                  \
    if (_e != hipSuccess) return ::ff::hip_status(_e, what); \
  } while (0)

#define FF_TRY(expr)               \
  do {                             \
    int _s = (expr);               \
    if (_s != FF_OK) return _s;    \
  } while (0)

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline size_t dtype_size(int dt) { return dt == FF_BF16 ? 2 : 4; }
inline size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ----------------------------------------------------------------- profiling
// Wraps one kernel launch: records events when profiling is enabled and
// checks the launch status.  `flops` / `bytes` are the launch's algorithmic
// work, accumulated per kernel name.
// Raises a kernel's dynamic-LDS limit to `bytes` on the current device, once per device (the
// attribute belongs to the device; `done` is the caller's per-kernel mask of device ordinals 0..63).
int ensure_smem_limit(const void* kernel, int bytes, std::atomic<uint64_t>& done);

// Brackets a launch with profiler events while profiling is on; a null name marks a launch that
// is never profiled (it records no events and allocates nothing).
struct LaunchScope {
  LaunchScope(const char* name, hipStream_t s, double flops, double bytes);
  ~LaunchScope();
  int status();   // FF_OK or FF_EHIP (checks hipGetLastError)
 private:
  const char* name_;
  hipStream_t stream_;
  double flops_, bytes_;
  int slot_;
};

// ----------------------------------------------------------------- workspace carving
struct Carver {
  char* base;
  size_t cap;
  size_t off = 0;
  Carver(void* b, size_t c) : base(static_cast<char*>(b)), cap(c) {}
  void* take(size_t bytes) {
    off = round_up(off, 256);
    void* p = base ? base + off : nullptr;
    off += bytes;
    return p;
  }
};

// ----------------------------------------------------------------- kernels (launchers)
// Per-sample streaming passes over [B, D] (SDE step, log-prob, losses): each sample's D
// elements are cut into `bps` chunks of `chunk` elements (a multiple of 2048), one block
// each, about 2048 blocks in all; per-block float64 partials are summed in a fixed order.
struct RowPlan {
  int64_t bps;     // blocks per sample
  int64_t chunk;   // elements per block
};
RowPlan row_plan(int64_t B, int64_t D);

// All launchers return FF_OK or FF_EHIP and expect validated arguments.

enum Epi : int {
  EPI_NONE = 0,       // out = acc + bias
  EPI_GELU = 1,       // out = gelu_tanh(acc + bias) for columns >= gelu_from, else acc + bias
  EPI_GATED = 2,      // out = resid + gate[b] * (acc + bias); gate null: out = resid + acc + bias
  EPI_QKV = 3,        // columns [Q | K | V] = [0, 3H) of acc + bias go through qk_norm_rope(*qkv) (fused when
                      // possible); columns from 3H on (N > 3H: a single-stream block's MLP input) take
                      // EPI_GELU's treatment with gelu_from = 3H and go to out
  EPI_SUMSQ = 5,      // out = acc + bias, and for columns [0, 2 sumsq_w) the sum of squares of each row's
                      // stored (rounded) values over every 64 columns: sumsq[m * (2 sumsq_w / 64) + n / 64]
                      // (the full-width Q / K RMS of a WAN block, added up in a fixed order by its reader)
};

struct QkvArgs;

struct GemmArgs {
  int dtype;
  int64_t M, N, K;
  // A = [A1 | A2] along K: A1 [M, K1] (lda1), A2 [M, K-K1] (lda2); K1 == K when A2 unused
  const void* A1; int64_t lda1; int64_t K1;
  const void* A2; int64_t lda2;
  const void* W; int64_t ldw;           // [N, K] row-major (nn.Linear weight)
  const void* bias;                     // [N] or null
  void* out; int64_t ldo;
  int epi;
  int64_t gelu_from;                    // EPI_GELU: first GELU column
  const float* gate; int64_t gate_ld;   // EPI_GATED: gate[(m / rows_per_sample) * gate_ld + n]
  const void* resid; int64_t ldr;       // EPI_GATED: residual (may alias out)
  int64_t rows_per_sample;
  const QkvArgs* qkv = nullptr;         // EPI_QKV: where Q, K and V^T go (out still names the packed
                                        // [Q | K | V] buffer, used when the fused path does not apply)
  // Scratch for split-K partial sums of a launch's last round (null: never split); see
  // gemm_split_bytes.  Launches on one stream may share it (each finishes before the next starts).
  void* split_ws = nullptr;
  size_t split_bytes = 0;
  float* sumsq = nullptr;               // EPI_SUMSQ: per-row partial sums of squares
  int64_t sumsq_w = 0;
};
// EPI_SUMSQ runs in the 256 x 256 tile kernel only: bf16, at least one tile per CU, N a multiple of
// 64 and 16-byte aligned rows, sumsq_w a multiple of 64 with 2 sumsq_w <= N.
bool gemm_sumsq_ok(const GemmArgs& a);
// Scratch bytes that let any launch split its last round: 255 tile partials of 256 KB and flags.
size_t gemm_split_bytes();
int gemm(const GemmArgs& a, hipStream_t s);
// Two GEMMs with the same epilogue kind, launched together when both are large bf16 problems.
int gemm2(const GemmArgs& a0, const GemmArgs& a1, hipStream_t s);

// out = epi(d_a[m] d_w[n] (A W^T)[m, n] + bias[n]): A [M, K] and W [N, K] OCP E4M3 codes (row
// strides lda, ldw in bytes = elements), d_a [M], d_w [N] float32 dequantisation scales, bias
// bf16 [N] or null, out bf16 [M, N]; epi EPI_NONE or EPI_GELU (from column gelu_from).
// K % 128 == 0; A, W 16-byte aligned with lda, ldw % 16 == 0.
struct Fp8GemmArgs {
  int64_t M, N, K;
  const void* A; int64_t lda; const float* d_a;
  const void* W; int64_t ldw; const float* d_w;
  const void* bias;
  void* out; int64_t ldo;
  int epi; int64_t gelu_from;
};
int gemm_fp8(const Fp8GemmArgs& a, hipStream_t s);

// Row quantisation to OCP E4M3: amax = max |x[r, :]|, codes = RNE(x * fl32(448 / amax)),
// d[r] = fl32(amax / 448) (zero rows: codes 0, d 0).  x of dtype [rows, cols] (stride ldx),
// q uint8 [rows, cols] (stride ldq); cols, ldx, ldq % 8 == 0, 16-byte aligned.
int quantize_fp8(int dtype, const void* x, int64_t ldx, void* q, int64_t ldq, float* d, int64_t rows, int64_t cols,
                 hipStream_t s);

// out[b, n] (+)= sum_k W[n, k] * act(in[b, k]) + bias[n]; in/out float32, W of dtype.
enum Act : int { ACT_NONE = 0, ACT_SILU = 1, ACT_GELU = 2 };
struct SkinnyArgs {
  int dtype;
  int64_t B, N, K;
  const float* in; int64_t ldi;
  int act_in;                 // activation applied to the input
  const void* W; const void* bias;
  float* out; int64_t ldo;
  int accumulate;             // 1: out += result
  int act_out;                // activation applied to the result (before accumulate)
  const int32_t* rowmap;      // row classes of `in` from row_classes (device), or null: all rows
};
int skinny_linear(const SkinnyArgs& a, hipStream_t s);
// The same input rows (a.in, a.B, a.K, activations, row map) against several weight matrices in as
// few launches as possible: segment i writes out_i [B, N_i] (row stride N_i).  a.W, a.bias, a.out,
// a.N and a.ldo are not used.
struct SkinnySeg {
  const void* W; const void* bias; float* out; int64_t N;
};
int skinny_linear_multi(const SkinnyArgs& a, const SkinnySeg* segs, int nseg, hipStream_t s);
// Classes of bitwise-equal rows of c [B, H] fp32 into map (device int32, row_classes_ints(B)
// entries), for skinny_linear to compute each distinct row once.
int64_t row_classes_ints(int64_t B);
int row_classes(const float* c, int64_t B, int64_t H, int32_t* map, hipStream_t s);

// y = Norm(x) * mul + add per row; row r belongs to sample r / rows_per_sample.
// mul = (1 + scale[b]) (if scale) * w (if w); add = shift[b] (if shift) + bias (if bias)
struct NormArgs {
  int dtype;
  int64_t rows, H;
  const void* x; int64_t ldx;
  void* y; int64_t ldy;
  int norm_kind; float eps;
  const float* shift; const float* scale; int64_t mod_ld;  // per-sample modulation (fp32)
  const void* w; const void* bias;                         // per-column affine (dtype)
  int64_t rows_per_sample;
};
int norm_modulate(const NormArgs& a, hipStream_t s);

// Streaming probe (mode 0 read, 1 write, 2 copy) over `chunks` 16-byte words; measurement only.
int stream_probe(int mode, bool nt, const void* src, void* dst, int64_t chunks, int blocks, hipStream_t s);

// Converts a float32 [rows, H] tensor to dtype (plain copy for F32) or dtype -> float32.
int cast_to_f32(int dtype, const void* in, float* out, int64_t n, hipStream_t s);

// Per-head QK RMSNorm + RoPE + relayout into the joint attention layout.
struct QkvArgs {
  int dtype;
  int64_t B, n_tok, tok_offset, n_joint;   // tokens of this stream, position in the joint sequence
  int64_t src_rows;                         // source rows per sample (token i of sample b is row b*src_rows+i)
  int heads, d;
  const void* q; const void* k; const void* v; int64_t ld;  // row stride of the packed source
  const void* q_w; const void* k_w;        // RMSNorm weights ([d] per-head, or [H] full-width)
  int full_width_norm;                      // 1: RMSNorm over all H before RoPE (WAN)
  int apply_norm;                           // 0: no QK norm (cross-attention V/K handled by caller)
  float eps;
  const float2* rope;                       // [n_tok - rope_from, d/2] (cos, sin) or null = no rotation
  int64_t rope_from;                        // tokens below it are not rotated; token i >= rope_from takes
                                            // table row i - rope_from (a joint text + image sequence)
  void* Q; void* Kd; void* Vt;              // Q, K [B, h, n_joint, d]; V transposed [B, h, d, n_joint]
  int v_transposed;
  // Full-width norm from precomputed sums (bf16, d = 128): per source row, sumsq_parts floats whose
  // first half adds up to the row's sum of q^2 over all H and second half to that of k^2 (EPI_SUMSQ).
  const float* sumsq = nullptr;
  int64_t sumsq_parts = 0;
};
int qk_norm_rope(const QkvArgs& a, hipStream_t s);

// (cos, sin) table for a (frames, rows, cols) grid: [N, d/2] float2, computed in float64.
int rope_table(float2* out, const int32_t grid[3], int d, const int32_t axes[3], double theta,
               hipStream_t s);

struct AttnArgs {
  int dtype;
  int64_t B, heads, d;
  int64_t n_q, n_kv;
  const void* Q; const void* K; const void* Vt;   // Q [B,h,n_q,d], K [B,h,n_kv,d], Vt [B,h,d,n_kv]
  // output split by query index: q < split -> out0 rows, else out1 rows (token-major, ld = H)
  void* out0; void* out1; int64_t split; int64_t ldo;
  float scale;
  // optional Q layout: element (b, h, q, :) at b*q_bs + h*q_hs + q*q_rs (all 0: [B, h, n_q, d])
  int64_t q_bs, q_hs, q_rs;
};
int attention(const AttnArgs& a, hipStream_t s);

// Gathers rows: out[b, j, :] = in[idx[b], j, :] (zero when idx out of range)
int gather_rows(int dtype, const void* in, const int32_t* idx, int64_t n_src, void* out,
                int64_t B, int64_t rows_per, int64_t width, hipStream_t s);

// temb input: [cos | sin](1000 t * 10000^(-j/128)) -> float32 [B, 256]
int timestep_sinusoid(const float* t, float* out, int64_t B, hipStream_t s);

// out[b, i, :] (+)= in (float32 [B, ld]) broadcast: used for WAN modulation tables
int add_table(const void* table, int dtype, const float* e, float* out, int64_t B, int64_t n,
              hipStream_t s);

}  // namespace ff
