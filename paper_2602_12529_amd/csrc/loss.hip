// Objectives that consume a rollout (include/ff_loss.h): forward noising,
// the AWM (Eq. 3) and DiffusionNFT (Eq. 2) losses, and the clipped-ratio GRPO
// objective on recomputed log-probabilities.
//
// The two matching losses are one streaming pass over [B, D] tensors (HBM
// bound): per sample, sum (a - (eps - x0))^2 (and the same for a second
// velocity), float32 within a thread's group of 8 elements and float64 from
// there on, in the fixed block / thread order of row_plan, then a per-sample
// finalize and a fixed-order mean.  The GRPO objective is a few thousand
// float64 elements: one workgroup.
#include <cmath>

#include "../../include/ff_loss.h"
#include "dev.h"
#include "ff_internal.h"

namespace ff {
namespace {

constexpr int kThreads = 256;
constexpr int64_t kVec = 8;

template <bool BF16, bool VEC>
__global__ __launch_bounds__(kThreads) void flow_noise_kernel(const void* __restrict__ x0, const void* __restrict__ eps,
                                                              const float* __restrict__ t, void* __restrict__ xt,
                                                              int64_t D) {
  const int64_t b = blockIdx.y;
  const float tb = t[b], sb = 1.0f - tb;
  const int64_t base = b * D;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads * (VEC ? kVec : 1);
  for (int64_t i = (static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x) * (VEC ? kVec : 1); i < D; i += stride) {
    if constexpr (VEC) {
      float xv[8], ev[8], out[8];
      ld8<BF16>(x0, base + i, xv);
      ld8<BF16>(eps, base + i, ev);
#pragma unroll
      for (int j = 0; j < 8; ++j) out[j] = fmaf(tb, ev[j], sb * xv[j]);
      st8<BF16>(xt, base + i, out);
    } else {
      st1<BF16>(xt, base + i, fmaf(tb, ld1<BF16>(eps, base + i), sb * ld1<BF16>(x0, base + i)));
    }
  }
}

// Per-block partial sums of (a - (eps - x0))^2 and, when TWO, of (a2 - (eps - x0))^2:
// partial[0][b][blk], partial[1][b][blk].
template <bool BF16, bool TWO, bool VEC>
__global__ __launch_bounds__(kThreads) void sqdist_kernel(const void* __restrict__ a, const void* __restrict__ a2,
                                                          const void* __restrict__ eps, const void* __restrict__ x0,
                                                          double* __restrict__ partial, int64_t B, int64_t D,
                                                          int64_t chunk) {
  const int64_t b = blockIdx.y;
  const int64_t base = b * D;
  const int64_t start = static_cast<int64_t>(blockIdx.x) * chunk;
  const int64_t end = start + chunk < D ? start + chunk : D;
  double acc1 = 0.0, acc2 = 0.0;
  if constexpr (VEC) {
    for (int64_t i = start + threadIdx.x * kVec; i < end; i += kThreads * kVec) {
      float av[8], ev[8], xv[8], bv[8];
      ld8<BF16>(a, base + i, av);
      ld8<BF16>(eps, base + i, ev);
      ld8<BF16>(x0, base + i, xv);
      if constexpr (TWO) ld8<BF16>(a2, base + i, bv);
      float p1 = 0.f, p2 = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float target = ev[j] - xv[j];
        const float d1 = av[j] - target;
        p1 = fmaf(d1, d1, p1);
        if constexpr (TWO) {
          const float d2 = bv[j] - target;
          p2 = fmaf(d2, d2, p2);
        }
      }
      acc1 += static_cast<double>(p1);
      if constexpr (TWO) acc2 += static_cast<double>(p2);
    }
  } else {
    for (int64_t i = start + threadIdx.x; i < end; i += kThreads) {
      const float target = ld1<BF16>(eps, base + i) - ld1<BF16>(x0, base + i);
      const float d1 = ld1<BF16>(a, base + i) - target;
      acc1 += static_cast<double>(d1 * d1);
      if constexpr (TWO) {
        const float d2 = ld1<BF16>(a2, base + i) - target;
        acc2 += static_cast<double>(d2 * d2);
      }
    }
  }
  __shared__ double red[2][kThreads / 64];
  acc1 = wave_sum(acc1);
  if constexpr (TWO) acc2 = wave_sum(acc2);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    red[0][wave] = acc1;
    red[1][wave] = acc2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double s1 = 0.0, s2 = 0.0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) {
      s1 += red[0][w];
      s2 += red[1][w];
    }
    const int64_t k = b * gridDim.x + blockIdx.x;
    partial[k] = s1;
    if constexpr (TWO) partial[B * gridDim.x + k] = s2;
  }
}

// per_sample[b] = w[b] * S1_b + (TWO ? (1 - w[b]) * S2_b : 0), S = fixed-order sums of the partials.
template <bool TWO>
__global__ __launch_bounds__(256) void loss_finalize(const double* __restrict__ partial, int64_t B, int64_t bps,
                                                     const float* __restrict__ w, double* __restrict__ per_sample) {
  __shared__ double red[2][256];
  const int64_t b = blockIdx.x;
  double s1 = 0.0, s2 = 0.0;
  for (int64_t i = threadIdx.x; i < bps; i += 256) {
    s1 += partial[b * bps + i];
    if constexpr (TWO) s2 += partial[(B + b) * bps + i];
  }
  red[0][threadIdx.x] = s1;
  red[1][threadIdx.x] = s2;
  __syncthreads();
  for (int k = 128; k > 0; k >>= 1) {
    if (threadIdx.x < k) {
      red[0][threadIdx.x] += red[0][threadIdx.x + k];
      red[1][threadIdx.x] += red[1][threadIdx.x + k];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const double wb = static_cast<double>(w[b]);
    per_sample[b] = TWO ? wb * red[0][0] + (1.0 - wb) * red[1][0] : wb * red[0][0];
  }
}

// loss = (sum_b per_sample[b]) / B, summed in a fixed order.
__global__ __launch_bounds__(256) void mean_kernel(const double* __restrict__ per_sample, int64_t B,
                                                   double* __restrict__ loss) {
  __shared__ double red[256];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < B; i += 256) s += per_sample[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int k = 128; k > 0; k >>= 1) {
    if (threadIdx.x < k) red[threadIdx.x] += red[threadIdx.x + k];
    __syncthreads();
  }
  if (threadIdx.x == 0) *loss = red[0] / static_cast<double>(B);
}

__global__ __launch_bounds__(256) void grpo_kernel(const double* __restrict__ lpn, const double* __restrict__ lpo,
                                                   const float* __restrict__ adv, const float* __restrict__ step_w,
                                                   int64_t B, int S, double clip_eps, double* __restrict__ loss,
                                                   int32_t* __restrict__ n_clipped) {
  __shared__ double red[256];
  __shared__ int cnt[256];
  const int64_t n = static_cast<int64_t>(S) * B;
  double s = 0.0;
  int c = 0;
  for (int64_t i = threadIdx.x; i < n; i += 256) {
    const int64_t k = i / B, b = i - k * B;
    const double r = exp(lpn[i] - lpo[i]);
    const double A = static_cast<double>(adv[b]);
    const double rc = r < 1.0 - clip_eps ? 1.0 - clip_eps : (r > 1.0 + clip_eps ? 1.0 + clip_eps : r);
    const double u = fmin(r * A, rc * A);
    s += (step_w ? static_cast<double>(step_w[k]) : 1.0) * u;
    c += (r < 1.0 - clip_eps || r > 1.0 + clip_eps) ? 1 : 0;
  }
  red[threadIdx.x] = s;
  cnt[threadIdx.x] = c;
  __syncthreads();
  for (int k = 128; k > 0; k >>= 1) {
    if (threadIdx.x < k) {
      red[threadIdx.x] += red[threadIdx.x + k];
      cnt[threadIdx.x] += cnt[threadIdx.x + k];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    *loss = -red[0] / static_cast<double>(n);
    if (n_clipped) *n_clipped = cnt[0];
  }
}

size_t loss_ws_bytes(int64_t B, int64_t D) {
  if (B == 0 || D == 0) return 0;
  return static_cast<size_t>(2 * B * row_plan(B, D).bps + B) * sizeof(double);
}

int check_rows(const char* fn, int32_t dtype, int64_t B, int64_t D) {
  if (dtype != FF_F32 && dtype != FF_BF16) return fail(FF_EINVAL, "%s: bad dtype %d", fn, dtype);
  if (B < 0 || D < 0) return fail(FF_EINVAL, "%s: negative shape B=%lld D=%lld", fn, (long long)B, (long long)D);
  if (B > 65535) return fail(FF_EUNSUPPORTED, "%s: B=%lld exceeds 65535", fn, (long long)B);
  return FF_OK;
}

// Shared body of ff_awm_loss (a2 == nullptr) and ff_nft_loss.
int matching_loss(const char* fn, const void* a, const void* a2, const void* eps, const void* x0, const float* w,
                  int64_t B, int64_t D, int32_t dtype, double* per_sample, double* loss, void* ws, size_t ws_bytes,
                  hipStream_t s) {
  FF_TRY(check_rows(fn, dtype, B, D));
  if (B == 0 || D == 0) return FF_OK;
  if (!a || !eps || !x0 || !w || !loss) return fail(FF_EINVAL, "%s: null pointer", fn);
  if (!aligned16(a) || !aligned16(eps) || !aligned16(x0) || (a2 && !aligned16(a2)))
    return fail(FF_EINVAL, "%s: tensor pointers must be 16-byte aligned", fn);
  const size_t want = loss_ws_bytes(B, D);
  if (!ws || ws_bytes < want)
    return fail(FF_EWORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, want, ws ? ws_bytes : 0);
  if (!aligned16(ws)) return fail(FF_EINVAL, "%s: workspace must be 16-byte aligned", fn);
  const RowPlan p = row_plan(B, D);
  double* partial = static_cast<double*>(ws);
  double* per = per_sample ? per_sample : partial + 2 * B * p.bps;
  const bool vec = D % kVec == 0, two = a2 != nullptr;
  const double esz = static_cast<double>(dtype_size(dtype));
  {
    LaunchScope ls(two ? "nft_loss" : "awm_loss", s, 0.0, static_cast<double>(B) * D * esz * (two ? 4.0 : 3.0));
    dim3 grid(static_cast<unsigned>(p.bps), static_cast<unsigned>(B));
#define FF_SQD(BF, TW, VC) \
  hipLaunchKernelGGL((sqdist_kernel<BF, TW, VC>), grid, dim3(kThreads), 0, s, a, a2, eps, x0, partial, B, D, p.chunk)
    if (dtype == FF_BF16) {
      if (two) { if (vec) FF_SQD(true, true, true); else FF_SQD(true, true, false); }
      else     { if (vec) FF_SQD(true, false, true); else FF_SQD(true, false, false); }
    } else {
      if (two) { if (vec) FF_SQD(false, true, true); else FF_SQD(false, true, false); }
      else     { if (vec) FF_SQD(false, false, true); else FF_SQD(false, false, false); }
    }
#undef FF_SQD
    FF_TRY(ls.status());
  }
  {
    LaunchScope ls("loss_finalize", s, 0.0, static_cast<double>(B) * p.bps * 8.0 * (two ? 2.0 : 1.0));
    if (two) hipLaunchKernelGGL(loss_finalize<true>, dim3(static_cast<unsigned>(B)), dim3(256), 0, s, partial, B, p.bps, w, per);
    else hipLaunchKernelGGL(loss_finalize<false>, dim3(static_cast<unsigned>(B)), dim3(256), 0, s, partial, B, p.bps, w, per);
    FF_TRY(ls.status());
    hipLaunchKernelGGL(mean_kernel, dim3(1), dim3(256), 0, s, per, B, loss);
    FF_TRY(ls.status());
  }
  return FF_OK;
}

}  // namespace
}  // namespace ff

using namespace ff;

extern "C" {

int ff_flow_noise(const void* x0, const void* eps, const float* t, void* xt, int64_t B, int64_t D, int32_t dtype,
                  void* stream) {
  const char* fn = "ff_flow_noise";
  FF_TRY(check_rows(fn, dtype, B, D));
  if (B == 0 || D == 0) return FF_OK;
  if (!x0 || !eps || !t || !xt) return fail(FF_EINVAL, "%s: null pointer", fn);
  if (xt == x0 || xt == eps) return fail(FF_EINVAL, "%s: xt aliases an input", fn);
  if (!aligned16(x0) || !aligned16(eps) || !aligned16(xt)) return fail(FF_EINVAL, "%s: pointers must be 16-byte aligned", fn);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool vec = D % kVec == 0;
  const int64_t per_block = kThreads * (vec ? kVec : 1);
  int64_t bx = (D + per_block - 1) / per_block;
  const int64_t cap = (4096 + B - 1) / B;
  if (bx > cap) bx = cap;
  if (bx < 1) bx = 1;
  dim3 grid(static_cast<unsigned>(bx), static_cast<unsigned>(B));
  LaunchScope ls("flow_noise", s, 0.0, static_cast<double>(B) * D * dtype_size(dtype) * 3.0);
  if (dtype == FF_BF16) {
    if (vec) hipLaunchKernelGGL((flow_noise_kernel<true, true>), grid, dim3(kThreads), 0, s, x0, eps, t, xt, D);
    else hipLaunchKernelGGL((flow_noise_kernel<true, false>), grid, dim3(kThreads), 0, s, x0, eps, t, xt, D);
  } else {
    if (vec) hipLaunchKernelGGL((flow_noise_kernel<false, true>), grid, dim3(kThreads), 0, s, x0, eps, t, xt, D);
    else hipLaunchKernelGGL((flow_noise_kernel<false, false>), grid, dim3(kThreads), 0, s, x0, eps, t, xt, D);
  }
  return ls.status();
}

int ff_loss_workspace_size(int64_t B, int64_t D, size_t* bytes) {
  if (!bytes) return fail(FF_EINVAL, "ff_loss_workspace_size: null output");
  if (B < 0 || D < 0) return fail(FF_EINVAL, "ff_loss_workspace_size: negative shape");
  *bytes = loss_ws_bytes(B, D);
  return FF_OK;
}

int ff_awm_loss(const void* v, const void* eps, const void* x0, const float* adv, int64_t B, int64_t D, int32_t dtype,
                double* per_sample, double* loss, void* workspace, size_t ws_bytes, void* stream) {
  return matching_loss("ff_awm_loss", v, nullptr, eps, x0, adv, B, D, dtype, per_sample, loss, workspace, ws_bytes,
                       static_cast<hipStream_t>(stream));
}

int ff_nft_loss(const void* v_pos, const void* v_neg, const void* eps, const void* x0, const float* r, int64_t B,
                int64_t D, int32_t dtype, double* per_sample, double* loss, void* workspace, size_t ws_bytes,
                void* stream) {
  if (!v_neg && B > 0 && D > 0) return fail(FF_EINVAL, "ff_nft_loss: null v_neg");
  return matching_loss("ff_nft_loss", v_pos, v_neg, eps, x0, r, B, D, dtype, per_sample, loss, workspace, ws_bytes,
                       static_cast<hipStream_t>(stream));
}

int ff_grpo_loss(const double* logp_new, const double* logp_old, const float* adv, const float* step_w, int64_t B,
                 int32_t S, double clip_eps, double* loss, int32_t* n_clipped, void* stream) {
  const char* fn = "ff_grpo_loss";
  if (B < 1 || S < 1) return fail(FF_EINVAL, "%s: need B >= 1 and S >= 1 (B=%lld S=%d)", fn, (long long)B, S);
  if (B > 65536 || static_cast<int64_t>(S) * B > 65536)
    return fail(FF_EUNSUPPORTED, "%s: S*B exceeds 65536 (B=%lld S=%d)", fn, (long long)B, S);
  if (!(clip_eps > 0.0) || !std::isfinite(clip_eps)) return fail(FF_EDOMAIN, "%s: clip_eps must be finite and > 0", fn);
  if (!logp_new || !logp_old || !adv || !loss) return fail(FF_EINVAL, "%s: null pointer", fn);
  hipStream_t s = static_cast<hipStream_t>(stream);
  LaunchScope ls("grpo_loss", s, 0.0, static_cast<double>(S) * B * 16.0);
  hipLaunchKernelGGL(grpo_kernel, dim3(1), dim3(256), 0, s, logp_new, logp_old, adv, step_w, B, S,
                     clip_eps, loss, n_clipped);
  return ls.status();
}

}  // extern "C"
