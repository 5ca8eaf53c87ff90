// Fused Flow-GRPO SDE step + transition log-probability (Sec. 3.1, Eq. 1) and
// group-normalised advantages (Sec. 2.3).
//
// SDE step: Eq. 1 is affine in (x, v) for fixed (t, dt, sigma):
//   mean = a x + b v,  a = 1 + sigma^2 dt / (2t),  b = dt (1 + sigma^2 (1-t) / (2t))
//   x_next = mean + c eps,  c = sigma sqrt(|dt|)
// a, b, c are formed on the host in float64 and passed as float32; the element
// work is one streaming pass over x, v, eps (HBM bound: 4 tensors x elem size
// per element).  The log-probability needs sum_d (x_next_stored - mean)^2 per
// sample: each thread accumulates 8 elements in float32, then float64 across
// groups, lanes, waves and blocks in a fixed order, so the result is bitwise
// reproducible and identical between ff_sde_step and ff_logprob.
#include <cmath>
#include <mutex>

#include "dev.h"
#include "ff_internal.h"

namespace ff {
namespace {

constexpr int kSdeThreads = 256;
constexpr int64_t kSdeVec = 8;

}  // namespace

RowPlan row_plan(int64_t B, int64_t D) {
  constexpr int64_t kTargetBlocks = 16384;   // 64 per CU: 16384 measured 12% faster than 2048 at 805 MB
  const int64_t per_pass = kSdeThreads * kSdeVec;
  int64_t want = (kTargetBlocks + B - 1) / B;
  int64_t max_blocks = (D + per_pass - 1) / per_pass;
  int64_t bps = want < max_blocks ? want : max_blocks;
  if (bps < 1) bps = 1;
  int64_t chunk = (D + bps - 1) / bps;
  chunk = (chunk + per_pass - 1) / per_pass * per_pass;
  bps = (D + chunk - 1) / chunk;
  return {bps, chunk};
}

namespace {

// Counter-based noise: Philox4x32-10 (Salmon et al., SC 2011) from its definition -- ten
// rounds of two 32x32 -> 64-bit products by 0xD2511F53 and 0xCD9E8D57 recombined with the
// other words and the round key, the key advancing by (0x9E3779B9, 0xBB67AE85) -- and the
// Box-Muller transform with u = (w + 1/2) 2^-32 in float32.  Element d of sample b in SDE
// step `step` is word d % 4 of the block with counter (d / 4 low, d / 4 high, b, step).
struct Ctr4 {
  uint32_t x, y, z, w;
};
__device__ __forceinline__ Ctr4 philox4x32_10(Ctr4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    // One 32 x 32 -> 64-bit product per multiplier gives both halves (v_mad_u64_u32: one
    // instruction instead of a mul_hi and a mul_lo; the step is ALU-bound on these).
    const uint64_t p0 = static_cast<uint64_t>(0xD2511F53u) * c.x, p1 = static_cast<uint64_t>(0xCD9E8D57u) * c.z;
    const uint32_t hi0 = static_cast<uint32_t>(p0 >> 32), lo0 = static_cast<uint32_t>(p0);
    const uint32_t hi1 = static_cast<uint32_t>(p1 >> 32), lo1 = static_cast<uint32_t>(p1);
    // Each three-way XOR is one v_bitop3_b32 (truth table 0x96 = a ^ b ^ c) instead of two XORs.
    const uint32_t x0 = static_cast<uint32_t>(__builtin_amdgcn_bitop3_b32(hi1, c.y, k0, 0x96));
    const uint32_t x2 = static_cast<uint32_t>(__builtin_amdgcn_bitop3_b32(hi0, c.w, k1, 0x96));
    c = {x0, lo1, x2, lo0};
  }
  return c;
}
// Box-Muller with the hardware transcendentals: v_log_f32 (log2) and v_sin_f32 / v_cos_f32,
// which take their angle in revolutions, so sin(2 pi u) is one instruction for u in (0, 1].
__device__ __forceinline__ void box_muller4(Ctr4 w, float* z) {
  constexpr float kInv32 = 2.3283064365386963e-10f;    // 2^-32
  constexpr float kM2Ln2 = -1.3862943611198906f;       // -2 ln 2: -2 ln u = kM2Ln2 log2 u
  const float u0 = (static_cast<float>(w.x) + 0.5f) * kInv32, u1 = (static_cast<float>(w.y) + 0.5f) * kInv32;
  const float u2 = (static_cast<float>(w.z) + 0.5f) * kInv32, u3 = (static_cast<float>(w.w) + 0.5f) * kInv32;
  const float r0 = __builtin_amdgcn_sqrtf(kM2Ln2 * __builtin_amdgcn_logf(u0));
  const float r1 = __builtin_amdgcn_sqrtf(kM2Ln2 * __builtin_amdgcn_logf(u2));
  z[0] = r0 * __builtin_amdgcn_cosf(u1);
  z[1] = r0 * __builtin_amdgcn_sinf(u1);
  z[2] = r1 * __builtin_amdgcn_cosf(u3);
  z[3] = r1 * __builtin_amdgcn_sinf(u3);
}
struct NoiseKey {
  uint32_t k0, k1, step;
};
// The four normals of Philox block n of sample b.
__device__ __forceinline__ void noise4(const NoiseKey& nk, uint32_t b, int64_t n, float* z) {
  const Ctr4 c{static_cast<uint32_t>(n), static_cast<uint32_t>(static_cast<uint64_t>(n) >> 32), b, nk.step};
  box_muller4(philox4x32_10(c, nk.k0, nk.k1), z);
}

// eps[b, d] of one SDE step, stored in the tensor's dtype.
template <bool BF16>
__global__ __launch_bounds__(256) void philox_normal_kernel(void* __restrict__ out, int64_t D, NoiseKey nk) {
  const int64_t b = blockIdx.y, nb = (D + 3) / 4;
  for (int64_t n = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; n < nb; n += static_cast<int64_t>(gridDim.x) * 256) {
    float z[4];
    noise4(nk, static_cast<uint32_t>(b), n, z);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (4 * n + j < D) st1<BF16>(out, b * D + 4 * n + j, z[j]);
  }
}

// Raw Philox words: block i has counter (base + i low, base + i high, c2, c3).
__global__ __launch_bounds__(256) void philox_words_kernel(uint32_t* __restrict__ out, int64_t n, uint64_t base,
                                                           uint32_t c2, uint32_t c3, uint32_t k0, uint32_t k1) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n; i += static_cast<int64_t>(gridDim.x) * 256) {
    const uint64_t ctr = base + static_cast<uint64_t>(i);
    const Ctr4 w = philox4x32_10({static_cast<uint32_t>(ctr), static_cast<uint32_t>(ctr >> 32), c2, c3}, k0, k1);
    out[4 * i] = w.x;
    out[4 * i + 1] = w.y;
    out[4 * i + 2] = w.z;
    out[4 * i + 3] = w.w;
  }
}

// One element: mean, stored next value, squared residual of the stored value.
template <bool BF16>
__device__ __forceinline__ float sde_elem(float x, float v, float e, float a, float b, float c,
                                          float& x_next) {
#pragma clang fp contract(off)
  float mean = fmaf(a, x, b * v);
  x_next = round_dt<BF16>(fmaf(c, e, mean));
  float r = x_next - mean;
  return r * r;
}

// MODE 0: SDE step (third = eps, writes x_next); MODE 1: log-prob only (third = x_next);
// MODE 2: SDE step with the noise generated from `nk` (third unused).
template <bool BF16, int MODE, bool LOGP, bool VEC>
__global__ __launch_bounds__(kSdeThreads) void sde_kernel(
    const void* __restrict__ x, const void* __restrict__ v, const void* __restrict__ third,
    void* __restrict__ x_next, double* __restrict__ partial, int64_t D, int64_t chunk, float a,
    float b, float c, NoiseKey nk) {
#pragma clang fp contract(off)
  const int64_t base = static_cast<int64_t>(blockIdx.y) * D;
  const int64_t start = static_cast<int64_t>(blockIdx.x) * chunk;
  const int64_t end = start + chunk < D ? start + chunk : D;
  double acc = 0.0;
  if constexpr (VEC) {
    // Two groups of 8 per thread per pass (loads of both issued first); the
    // chunk is a multiple of 2 * 256 * 8 elements except possibly at the end
    // of the sample, where the second group is skipped.
    for (int64_t i = start + threadIdx.x * kSdeVec; i < end; i += 2 * kSdeThreads * kSdeVec) {
      const int64_t i2 = i + kSdeThreads * kSdeVec;
      const bool two = i2 < end;
      float xv[2][8], vv[2][8], tv[2][8], out[8];
      ld8_nt<BF16>(x, base + i, xv[0]);
      ld8_nt<BF16>(v, base + i, vv[0]);
      if constexpr (MODE != 2) ld8_nt<BF16>(third, base + i, tv[0]);
      if (two) {
        ld8_nt<BF16>(x, base + i2, xv[1]);
        ld8_nt<BF16>(v, base + i2, vv[1]);
        if constexpr (MODE != 2) ld8_nt<BF16>(third, base + i2, tv[1]);
      }
      if constexpr (MODE == 2) {
        // i and i2 are multiples of 8 within the sample: two whole Philox blocks each
        noise4(nk, blockIdx.y, i >> 2, tv[0]);
        noise4(nk, blockIdx.y, (i >> 2) + 1, tv[0] + 4);
        if (two) {
          noise4(nk, blockIdx.y, i2 >> 2, tv[1]);
          noise4(nk, blockIdx.y, (i2 >> 2) + 1, tv[1] + 4);
        }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        if (h == 1 && !two) break;
        float part = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          if constexpr (MODE != 1) {
            float r2 = sde_elem<BF16>(xv[h][j], vv[h][j], tv[h][j], a, b, c, out[j]);
            part = part + r2;
          } else {
            float mean = fmaf(a, xv[h][j], b * vv[h][j]);
            float r = tv[h][j] - mean;
            part = part + r * r;
          }
        }
        if constexpr (MODE != 1) st8_nt<BF16>(x_next, base + (h == 0 ? i : i2), out);
        if constexpr (LOGP) acc += static_cast<double>(part);
      }
    }
  } else {
    for (int64_t i = start + threadIdx.x; i < end; i += kSdeThreads) {
      float xv = ld1<BF16>(x, base + i), vv = ld1<BF16>(v, base + i), tv;
      if constexpr (MODE == 2) {
        float z[4];
        noise4(nk, blockIdx.y, i >> 2, z);
        tv = z[i & 3];
      } else {
        tv = ld1<BF16>(third, base + i);
      }
      float r2;
      if constexpr (MODE != 1) {
        float out;
        r2 = sde_elem<BF16>(xv, vv, tv, a, b, c, out);
        st1<BF16>(x_next, base + i, out);
      } else {
        float mean = fmaf(a, xv, b * vv);
        float r = tv - mean;
        r2 = r * r;
      }
      if constexpr (LOGP) acc += static_cast<double>(r2);
    }
  }
  if constexpr (LOGP) {
    __shared__ double red[kSdeThreads / 64];
    acc = wave_sum(acc);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) red[wave] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
      double s = 0.0;
#pragma unroll
      for (int w = 0; w < kSdeThreads / 64; ++w) s += red[w];
      partial[static_cast<int64_t>(blockIdx.y) * gridDim.x + blockIdx.x] = s;
    }
  }
}

// logp[b] = -S_b / (2 c^2) + const, S_b = fixed-order sum of the sample's block partials.
__global__ __launch_bounds__(256) void logp_finalize(const double* __restrict__ partial, int64_t bps,
                                                     double* __restrict__ logp, double inv_2var,
                                                     double cst) {
  __shared__ double red[256];
  const int64_t b = blockIdx.x;
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < bps; i += 256) s += partial[b * bps + i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) logp[b] = -red[0] * inv_2var + cst;
}

template <int MODE>
int launch_sde(int dtype, const void* x, const void* v, const void* third, void* x_next, double* logp,
               int64_t B, int64_t D, float a, float b, float c, double inv_2var, double cst,
               void* ws, hipStream_t s, NoiseKey nk = {0, 0, 0}, bool profile = true) {
  RowPlan p = row_plan(B, D);
  dim3 grid(static_cast<unsigned>(p.bps), static_cast<unsigned>(B));
  double* partial = static_cast<double*>(ws);
  const bool vec = (D % kSdeVec) == 0;
  const bool lp = logp != nullptr;
  const double esz = static_cast<double>(dtype_size(dtype));
  const double bytes = static_cast<double>(B) * D * esz * (MODE == 0 ? 4.0 : 3.0);
  {
    LaunchScope ls(!profile ? nullptr : (MODE == 0 ? "sde_step" : (MODE == 2 ? "sde_step_philox" : "logprob")), s,
                   0.0, bytes);
#define FF_SDE_LAUNCH(BF, LP, VC)                                                                 \
  hipLaunchKernelGGL((sde_kernel<BF, MODE, LP, VC>), grid, dim3(kSdeThreads), 0, s, x, v, third, \
                     x_next, partial, D, p.chunk, a, b, c, nk)
    if (dtype == FF_BF16) {
      if (lp) { if (vec) FF_SDE_LAUNCH(true, true, true); else FF_SDE_LAUNCH(true, true, false); }
      else    { if (vec) FF_SDE_LAUNCH(true, false, true); else FF_SDE_LAUNCH(true, false, false); }
    } else {
      if (lp) { if (vec) FF_SDE_LAUNCH(false, true, true); else FF_SDE_LAUNCH(false, true, false); }
      else    { if (vec) FF_SDE_LAUNCH(false, false, true); else FF_SDE_LAUNCH(false, false, false); }
    }
#undef FF_SDE_LAUNCH
    FF_TRY(ls.status());
  }
  if (lp) {
    LaunchScope ls(profile ? "logp_finalize" : nullptr, s, 0.0, static_cast<double>(B) * p.bps * 8.0);
    hipLaunchKernelGGL(logp_finalize, dim3(static_cast<unsigned>(B)), dim3(256), 0, s, partial, p.bps,
                       logp, inv_2var, cst);
    FF_TRY(ls.status());
  }
  return FF_OK;
}

int check_sde_args(const char* fn, const void* x, const void* v, const void* third, const void* out,
                   int64_t B, int64_t D, double t, double t_next, double sigma, int32_t dtype) {
  if (dtype != FF_F32 && dtype != FF_BF16) return fail(FF_EINVAL, "%s: bad dtype %d", fn, dtype);
  if (B < 0 || D < 0) return fail(FF_EINVAL, "%s: negative shape B=%lld D=%lld", fn, (long long)B, (long long)D);
  if (B > 65535) return fail(FF_EUNSUPPORTED, "%s: B=%lld exceeds 65535", fn, (long long)B);
  if (!std::isfinite(t) || !std::isfinite(t_next) || !std::isfinite(sigma))
    return fail(FF_EDOMAIN, "%s: non-finite t/t_next/sigma", fn);
  if (!(t_next < t) || t > 1.0 || t_next < 0.0)
    return fail(FF_EDOMAIN, "%s: need 0 <= t_next < t <= 1 (t=%g, t_next=%g)", fn, t, t_next);
  if (sigma < 0.0) return fail(FF_EDOMAIN, "%s: sigma=%g < 0", fn, sigma);
  if (sigma > 0.0 && !(t > 0.0)) return fail(FF_EDOMAIN, "%s: sigma > 0 needs t > 0", fn);
  if (B == 0 || D == 0) return FF_OK;
  if (!x || !v || !third || (out == nullptr && third == nullptr))
    return fail(FF_EINVAL, "%s: null tensor pointer", fn);
  if (!aligned16(x) || !aligned16(v) || !aligned16(third) || (out && !aligned16(out)))
    return fail(FF_EINVAL, "%s: tensor pointers must be 16-byte aligned", fn);
  return FF_OK;
}

int check_ws(const char* fn, int64_t B, int64_t D, bool need, const void* ws, size_t ws_bytes) {
  if (!need) return FF_OK;
  size_t want = static_cast<size_t>(B) * row_plan(B, D).bps * sizeof(double);
  if (!ws || ws_bytes < want)
    return fail(FF_EWORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, want, ws ? ws_bytes : 0);
  if (!aligned16(ws)) return fail(FF_EINVAL, "%s: workspace must be 16-byte aligned", fn);
  return FF_OK;
}

struct Coef {
  float a, b, c;
  double inv_2var, cst;
};

Coef coefficients(double t, double t_next, double sigma, int64_t D) {
  const double dt = t_next - t;
  Coef k{};
  if (sigma == 0.0) {
    k.a = 1.0f;
    k.b = static_cast<float>(dt);
    k.c = 0.0f;
    return k;
  }
  const double s2 = sigma * sigma;
  k.a = static_cast<float>(1.0 + s2 * dt / (2.0 * t));
  k.b = static_cast<float>(dt * (1.0 + s2 * (1.0 - t) / (2.0 * t)));
  const double std = sigma * std::sqrt(-dt);
  k.c = static_cast<float>(std);
  k.inv_2var = 1.0 / (2.0 * std * std);
  k.cst = -static_cast<double>(D) * (std::log(std) + 0.5 * std::log(2.0 * M_PI));
  return k;
}

// Allocation-free variant: the per-block float64 partial sums of the log-probability live in a
// file-scope device array instead of a caller workspace.  B x blocks-per-sample never exceeds
// max(B, 16383 + B) (the row plan aims at 16384 blocks in all, one per sample at least), so
// 81920 doubles (640 KiB per device) cover every B <= 65535.
constexpr int64_t kScratchDoubles = 81920;
__device__ __align__(256) double scratch[kScratchDoubles];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
double* g_scratch_dev[kMaxDevices] = {};

// The current device's address of `scratch`, looked up once per device with that device current
// (the host-side symbol is not a device address; each device holds its own copy of the array).
int scratch_address(double** out) {
  int dev = 0;
  FF_CHECK_HIP(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(FF_EUNSUPPORTED, "device ordinal %d above %d", dev, kMaxDevices - 1);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    FF_CHECK_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (!p) return fail(FF_EHIP, "hipGetSymbolAddress(scratch) returned null");
    g_scratch_dev[dev] = static_cast<double*>(p);
  }
  *out = g_scratch_dev[dev];
  return FF_OK;
}

}  // namespace
}  // namespace ff

using namespace ff;

extern "C" {

int ff_sde_workspace_size(int64_t B, int64_t D, size_t* bytes) {
  if (!bytes) return fail(FF_EINVAL, "ff_sde_workspace_size: null output");
  if (B < 0 || D < 0) return fail(FF_EINVAL, "ff_sde_workspace_size: negative shape");
  *bytes = (B == 0 || D == 0) ? 0 : static_cast<size_t>(B) * row_plan(B, D).bps * sizeof(double);
  return FF_OK;
}

// D = 0: every sample is an empty vector, whose log-density (an empty sum, no normalising terms)
// is 0; nothing else is read or written.
__global__ __launch_bounds__(256) void zero_logp_kernel(double* __restrict__ logp, int64_t B) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < B) logp[i] = 0.0;
}
int zero_logp(const char* fn, double* logp, int64_t B, void* stream, bool profile = true) {
  if (!logp) return FF_OK;
  if ((reinterpret_cast<uintptr_t>(logp) & 7u) != 0) return fail(FF_EINVAL, "%s: logp misaligned", fn);
  hipStream_t s = static_cast<hipStream_t>(stream);
  LaunchScope ls(profile ? "logp_zero" : nullptr, s, 0.0, 8.0 * static_cast<double>(B));
  hipLaunchKernelGGL(zero_logp_kernel, dim3(static_cast<unsigned>((B + 255) / 256)), dim3(256), 0, s, logp, B);
  return ls.status();
}

int ff_sde_step(const void* x, const void* v, const void* eps, void* x_next, double* logp, int64_t B,
                int64_t D, double t, double t_next, double sigma, int32_t dtype, void* workspace,
                size_t ws_bytes, void* stream) {
  FF_TRY(check_sde_args("ff_sde_step", x, v, eps, x_next, B, D, t, t_next, sigma, dtype));
  if (sigma == 0.0 && logp) return fail(FF_EDOMAIN, "ff_sde_step: an ODE step (sigma=0) has no log-probability");
  if (B == 0) return FF_OK;
  if (D == 0) return zero_logp("ff_sde_step", logp, B, stream);
  if (!x_next) return fail(FF_EINVAL, "ff_sde_step: null x_next");
  if (x_next == x || x_next == v || x_next == eps) return fail(FF_EINVAL, "ff_sde_step: x_next aliases an input");
  if (logp && !aligned16(logp)) { /* doubles need 8-byte alignment only */
    if ((reinterpret_cast<uintptr_t>(logp) & 7u) != 0) return fail(FF_EINVAL, "ff_sde_step: logp misaligned");
  }
  FF_TRY(check_ws("ff_sde_step", B, D, logp != nullptr, workspace, ws_bytes));
  Coef k = coefficients(t, t_next, sigma, D);
  return launch_sde<0>(dtype, x, v, eps, x_next, logp, B, D, k.a, k.b, k.c, k.inv_2var, k.cst, workspace,
                       static_cast<hipStream_t>(stream));
}

int ff_sde_step_noalloc(const void* x, const void* v, const void* eps, void* x_next, double* logp, int64_t B,
                        int64_t D, double t, double t_next, double sigma, int32_t dtype, void* stream) {
  const char* fn = "ff_sde_step_noalloc";
  FF_TRY(check_sde_args(fn, x, v, eps, x_next, B, D, t, t_next, sigma, dtype));
  if (sigma == 0.0 && logp) return fail(FF_EDOMAIN, "%s: an ODE step (sigma=0) has no log-probability", fn);
  if (B == 0) return FF_OK;
  if (D == 0) return zero_logp(fn, logp, B, stream, /*profile=*/false);
  if (!x_next) return fail(FF_EINVAL, "%s: null x_next", fn);
  if (x_next == x || x_next == v || x_next == eps) return fail(FF_EINVAL, "%s: x_next aliases an input", fn);
  if (logp && (reinterpret_cast<uintptr_t>(logp) & 7u) != 0) return fail(FF_EINVAL, "%s: logp misaligned", fn);
  double* partial = nullptr;
  if (logp) {
    const int64_t need = B * row_plan(B, D).bps;
    if (need > kScratchDoubles)
      return fail(FF_EUNSUPPORTED, "%s: %lld partial sums exceed the %lld-entry scratch", fn, (long long)need,
                  (long long)kScratchDoubles);
    FF_TRY(scratch_address(&partial));
  }
  Coef k = coefficients(t, t_next, sigma, D);
  return launch_sde<0>(dtype, x, v, eps, x_next, logp, B, D, k.a, k.b, k.c, k.inv_2var, k.cst, partial,
                       static_cast<hipStream_t>(stream), NoiseKey{0, 0, 0}, /*profile=*/false);
}

int ff_logprob(const void* x, const void* v, const void* x_next, double* logp, int64_t B, int64_t D,
               double t, double t_next, double sigma, int32_t dtype, void* workspace, size_t ws_bytes,
               void* stream) {
  FF_TRY(check_sde_args("ff_logprob", x, v, x_next, nullptr, B, D, t, t_next, sigma, dtype));
  if (!(sigma > 0.0)) return fail(FF_EDOMAIN, "ff_logprob: needs sigma > 0");
  if (B == 0) return FF_OK;
  if (!logp) return fail(FF_EINVAL, "ff_logprob: null logp");
  if (D == 0) return zero_logp("ff_logprob", logp, B, stream);
  if ((reinterpret_cast<uintptr_t>(logp) & 7u) != 0) return fail(FF_EINVAL, "ff_logprob: logp misaligned");
  FF_TRY(check_ws("ff_logprob", B, D, true, workspace, ws_bytes));
  Coef k = coefficients(t, t_next, sigma, D);
  return launch_sde<1>(dtype, x, v, x_next, nullptr, logp, B, D, k.a, k.b, k.c, k.inv_2var, k.cst,
                       workspace, static_cast<hipStream_t>(stream));
}

int ff_sde_step_philox(const void* x, const void* v, void* x_next, double* logp, int64_t B, int64_t D, double t,
                       double t_next, double sigma, uint64_t seed, uint32_t step, int32_t dtype, void* workspace,
                       size_t ws_bytes, void* stream) {
  const char* fn = "ff_sde_step_philox";
  FF_TRY(check_sde_args(fn, x, v, x, x_next, B, D, t, t_next, sigma, dtype));
  if (sigma == 0.0 && logp) return fail(FF_EDOMAIN, "%s: an ODE step (sigma=0) has no log-probability", fn);
  if (B == 0) return FF_OK;
  if (D == 0) return zero_logp(fn, logp, B, stream);
  if (!x_next) return fail(FF_EINVAL, "%s: null x_next", fn);
  if (x_next == x || x_next == v) return fail(FF_EINVAL, "%s: x_next aliases an input", fn);
  if (logp && (reinterpret_cast<uintptr_t>(logp) & 7u) != 0) return fail(FF_EINVAL, "%s: logp misaligned", fn);
  FF_TRY(check_ws(fn, B, D, logp != nullptr, workspace, ws_bytes));
  Coef k = coefficients(t, t_next, sigma, D);
  const NoiseKey nk{static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32), step};
  return launch_sde<2>(dtype, x, v, nullptr, x_next, logp, B, D, k.a, k.b, k.c, k.inv_2var, k.cst, workspace,
                       static_cast<hipStream_t>(stream), nk);
}

int ff_philox_normal(void* eps, int64_t B, int64_t D, uint64_t seed, uint32_t step, int32_t dtype, void* stream) {
  const char* fn = "ff_philox_normal";
  if (dtype != FF_F32 && dtype != FF_BF16) return fail(FF_EINVAL, "%s: bad dtype %d", fn, dtype);
  if (B < 0 || D < 0) return fail(FF_EINVAL, "%s: negative shape", fn);
  if (B > 65535) return fail(FF_EUNSUPPORTED, "%s: B=%lld exceeds 65535", fn, (long long)B);
  if (B == 0 || D == 0) return FF_OK;
  if (!eps) return fail(FF_EINVAL, "%s: null eps", fn);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const NoiseKey nk{static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32), step};
  const int64_t nb = (D + 3) / 4;
  int64_t bx = (nb + 255) / 256;
  const int64_t cap = (2048 + B - 1) / B;
  if (bx > cap) bx = cap;
  dim3 grid(static_cast<unsigned>(bx), static_cast<unsigned>(B));
  LaunchScope ls("philox_normal", s, 0.0, static_cast<double>(B) * D * dtype_size(dtype));
  if (dtype == FF_BF16) hipLaunchKernelGGL(philox_normal_kernel<true>, grid, dim3(256), 0, s, eps, D, nk);
  else hipLaunchKernelGGL(philox_normal_kernel<false>, grid, dim3(256), 0, s, eps, D, nk);
  return ls.status();
}

int ff_philox4x32(uint32_t* out, int64_t n, uint64_t ctr_base, uint32_t c2, uint32_t c3, uint64_t key,
                  void* stream) {
  const char* fn = "ff_philox4x32";
  if (n < 0) return fail(FF_EINVAL, "%s: negative count", fn);
  if (n == 0) return FF_OK;
  if (!out) return fail(FF_EINVAL, "%s: null out", fn);
  hipStream_t s = static_cast<hipStream_t>(stream);
  int64_t bx = (n + 255) / 256;
  if (bx > 4096) bx = 4096;
  LaunchScope ls("philox4x32", s, 0.0, static_cast<double>(n) * 16.0);
  hipLaunchKernelGGL(philox_words_kernel, dim3(static_cast<unsigned>(bx)), dim3(256), 0, s, out, n, ctr_base, c2, c3,
                     static_cast<uint32_t>(key), static_cast<uint32_t>(key >> 32));
  return ls.status();
}

}  // extern "C"

// ------------------------------------------------------------------ advantages
namespace ff {
namespace {

constexpr int kAdvThreads = 256;
constexpr int kAdvMaxK = 16;
constexpr int kAdvMaxStats = 4096;

// Value j of sample i: the weighted reward sum (mode 0, j = 0) or reward j (mode 1).
__device__ __forceinline__ double adv_value(const float* r, const float* w, int64_t i, int K, int mode, int j) {
  if (mode == 1) return static_cast<double>(r[i * K + j]);
  double s = 0.0;
  for (int k = 0; k < K; ++k) s += static_cast<double>(w ? w[k] : 1.0f) * static_cast<double>(r[i * K + k]);
  return s;
}

__global__ __launch_bounds__(kAdvThreads) void group_adv_kernel(const float* __restrict__ rewards,
                                                                const float* __restrict__ weights,
                                                                const int32_t* __restrict__ gid, int64_t N, int K,
                                                                int G, int mode, float eps, float* __restrict__ adv,
                                                                int32_t* __restrict__ counts) {
  extern __shared__ double stats[];          // [G * KK] means, then [G * KK] denominators
  const int KK = mode == 1 ? K : 1;
  double* s_mean = stats;
  double* s_den = stats + static_cast<int64_t>(G) * KK;
  for (int g = threadIdx.x; g < G; g += kAdvThreads) {
    int32_t cnt = 0;
    for (int64_t i = 0; i < N; ++i) cnt += (gid[i] == g) ? 1 : 0;
    if (counts) counts[g] = cnt;
    for (int j = 0; j < KK; ++j) {
      double sum = 0.0;
      for (int64_t i = 0; i < N; ++i)
        if (gid[i] == g) sum += adv_value(rewards, weights, i, K, mode, j);
      double mean = cnt ? sum / cnt : 0.0;
      double ss = 0.0;
      for (int64_t i = 0; i < N; ++i)
        if (gid[i] == g) {
          double d = adv_value(rewards, weights, i, K, mode, j) - mean;
          ss += d * d;
        }
      double sd = cnt ? sqrt(ss / cnt) : 0.0;
      s_mean[g * KK + j] = mean;
      s_den[g * KK + j] = sd + static_cast<double>(eps);
    }
  }
  __syncthreads();
  for (int64_t i = threadIdx.x; i < N; i += kAdvThreads) {
    const int g = gid[i];
    if (g < 0 || g >= G) {
      adv[i] = __int_as_float(0x7fc00000);
      continue;
    }
    double a = 0.0;
    if (mode == 1) {
      for (int j = 0; j < K; ++j) {
        double w = weights ? static_cast<double>(weights[j]) : 1.0;
        a += w * (static_cast<double>(rewards[i * K + j]) - s_mean[g * K + j]) / s_den[g * K + j];
      }
    } else {
      double val = adv_value(rewards, weights, i, K, 0, 0);
      a = (val - s_mean[g]) / s_den[g];
    }
    adv[i] = static_cast<float>(a);
  }
}

}  // namespace
}  // namespace ff

extern "C" int ff_group_advantage(const float* rewards, const float* weights, const int32_t* group_id,
                                  int64_t N, int32_t K, int32_t n_groups, int32_t mode, float eps, float* adv,
                                  int32_t* group_count, void* stream) {
  const char* fn = "ff_group_advantage";
  if (N < 0) return fail(FF_EINVAL, "%s: negative N", fn);
  if (N > (int64_t(1) << 20)) return fail(FF_EUNSUPPORTED, "%s: N=%lld above 2^20 samples", fn, (long long)N);
  if (K < 1 || K > kAdvMaxK) return fail(FF_EUNSUPPORTED, "%s: K=%d outside [1, %d]", fn, K, kAdvMaxK);
  if (n_groups < 1) return fail(FF_EINVAL, "%s: n_groups=%d < 1", fn, n_groups);
  if (mode != 0 && mode != 1) return fail(FF_EINVAL, "%s: mode=%d", fn, mode);
  const int KK = mode == 1 ? K : 1;
  if (static_cast<int64_t>(n_groups) * KK > kAdvMaxStats)
    return fail(FF_EUNSUPPORTED, "%s: n_groups*K=%lld exceeds %d", fn, (long long)n_groups * KK, kAdvMaxStats);
  if (!std::isfinite(eps) || eps < 0.f) return fail(FF_EDOMAIN, "%s: eps must be finite and >= 0", fn);
  if (N == 0 && !group_count) return FF_OK;
  if (N > 0 && (!rewards || !group_id || !adv)) return fail(FF_EINVAL, "%s: null tensor pointer", fn);
  hipStream_t s = static_cast<hipStream_t>(stream);
  LaunchScope ls("group_advantage", s, 0.0, static_cast<double>(N) * (4.0 * K + 8.0));
  size_t shm = static_cast<size_t>(n_groups) * KK * 2 * sizeof(double);
  hipLaunchKernelGGL(group_adv_kernel, dim3(1), dim3(kAdvThreads), shm, s, rewards, weights, group_id, N, K,
                     n_groups, mode, eps, adv, group_count);
  return ls.status();
}
