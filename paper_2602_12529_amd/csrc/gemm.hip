// Y = A W^T (+ epilogue) for the DiT's linear layers: QKV, output, MLP, embedders.
//
// bf16: MFMA 32x32x16 (gfx950) tiles, fp32 accumulation.  A [M, K] and W [N, K]
// are both K-contiguous (nn.Linear layout).  A workgroup computes a BM x BN
// tile; its waves split it into wave tiles of (BM/WAVES_M) x (BN/WAVES_N),
// each a grid of 32x32 MFMA blocks.  K advances in slabs of 64 that are
// staged global -> registers -> LDS with two LDS buffers (the next slab's
// global loads are in flight while the current slab is multiplied).  Each
// 128-byte LDS row holds 8 chunks of 16 bytes stored at chunk ^ (row & 7), so
// the 16-byte fragment reads of 8 consecutive rows hit distinct banks.
// Tiles are ordered so that consecutive tiles of one XCD (workgroups are
// dealt round-robin over the 8 XCDs) share A rows in that XCD's L2.
//
// Epilogues fuse the bias, GELU-tanh (from a column on, for the fused
// single-stream projection) and the adaLN-gated residual X + g * (.).
//
// f32: a plain LDS-tiled FMA kernel with the same epilogues, for the float32
// configurations.
#include "dev.h"
#include "ff_internal.h"

namespace ff {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

struct GemmParams {
  int64_t M, N, K;
  const void* A1; int64_t lda1; int64_t K1;
  const void* A2; int64_t lda2;
  const void* W; int64_t ldw;
  const void* bias;
  void* out; int64_t ldo;
  int64_t gelu_from;
  const float* gate; int64_t gate_ld;
  const void* resid; int64_t ldr;
  int64_t rows_per_sample;
};

template <bool BF16, int EPI>
__device__ __forceinline__ void epi_store(const GemmParams& p, int64_t m, int64_t n, float acc) {
  float v = acc;
  if (p.bias) v += ld1<BF16>(p.bias, n);
  if constexpr (EPI == EPI_GELU) {
    if (n >= p.gelu_from) v = gelu_tanh_f(v);
  } else if constexpr (EPI == EPI_GATED) {
    const float g = p.gate[(m / p.rows_per_sample) * p.gate_ld + n];
    v = ld1<BF16>(p.resid, m * p.ldr + n) + g * v;
  }
  st1<BF16>(p.out, m * p.ldo + n, v);
}

// Maps the linear workgroup id to a (tile_m, tile_n) pair: first regroup ids
// so each XCD owns a contiguous range, then walk GROUP_M tile rows at a time.
__device__ __forceinline__ void tile_coords(int64_t pid, int64_t num_m, int64_t num_n, int64_t& tm,
                                            int64_t& tn) {
  const int64_t total = num_m * num_n;
  const int64_t full = total / 8 * 8;
  int64_t lid = pid;
  if (pid < full) lid = (pid % 8) * (full / 8) + pid / 8;
  constexpr int64_t GROUP_M = 8;
  const int64_t in_group = GROUP_M * num_n;
  const int64_t gidx = lid / in_group;
  const int64_t first_m = gidx * GROUP_M;
  const int64_t gsize = (num_m - first_m) < GROUP_M ? (num_m - first_m) : GROUP_M;
  const int64_t r = lid % in_group;
  tm = first_m + r % gsize;
  tn = r / gsize;
}

constexpr int BK = 64;

template <int BM, int BN, int WAVES_M, int WAVES_N, int EPI>
__global__ __launch_bounds__(WAVES_M* WAVES_N * 64, 1) void gemm_bf16_kernel(GemmParams p) {
  constexpr int THREADS = WAVES_M * WAVES_N * 64;
  constexpr int TM = BM / WAVES_M, TN = BN / WAVES_N;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int A_LOADS = BM * 8 / THREADS, B_LOADS = BN * 8 / THREADS;
  static_assert(A_LOADS * THREADS == BM * 8 && B_LOADS * THREADS == BN * 8, "tile/threads mismatch");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  constexpr int STAGE = (BM + BN) * BK * 2;

  const int64_t num_m = (p.M + BM - 1) / BM, num_n = (p.N + BN - 1) / BN;
  int64_t tm, tn;
  tile_coords(blockIdx.x, num_m, num_n, tm, tn);
  const int64_t m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;

  // Global source rows/chunks of this thread (fixed across K).
  const bf16_t* A1 = static_cast<const bf16_t*>(p.A1);
  const bf16_t* A2 = static_cast<const bf16_t*>(p.A2);
  const bf16_t* Wp = static_cast<const bf16_t*>(p.W);
  int a_row[A_LOADS], b_row[B_LOADS];
  int64_t a_grow[A_LOADS], b_grow[B_LOADS];
  const int chunk = tid & 7;
#pragma unroll
  for (int i = 0; i < A_LOADS; ++i) {
    a_row[i] = (tid + i * THREADS) >> 3;
    int64_t g = m0 + a_row[i];
    a_grow[i] = g < p.M ? g : p.M - 1;
  }
#pragma unroll
  for (int i = 0; i < B_LOADS; ++i) {
    b_row[i] = (tid + i * THREADS) >> 3;
    int64_t g = n0 + b_row[i];
    b_grow[i] = g < p.N ? g : p.N - 1;
  }

  uint4 ra[A_LOADS], rb[B_LOADS];
  auto load_slab = [&](int64_t k0) {
    const bf16_t* src;
    int64_t ld, kc;
    if (k0 < p.K1) { src = A1; ld = p.lda1; kc = k0; }
    else { src = A2; ld = p.lda2; kc = k0 - p.K1; }
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i)
      ra[i] = *reinterpret_cast<const uint4*>(src + a_grow[i] * ld + kc + chunk * 8);
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i)
      rb[i] = *reinterpret_cast<const uint4*>(Wp + b_grow[i] * p.ldw + k0 + chunk * 8);
  };
  auto store_slab = [&](int buf) {
    char* As = smem + buf * STAGE;
    char* Bs = As + BM * BK * 2;
#pragma unroll
    for (int i = 0; i < A_LOADS; ++i)
      *reinterpret_cast<uint4*>(As + a_row[i] * 128 + ((chunk ^ (a_row[i] & 7)) << 4)) = ra[i];
#pragma unroll
    for (int i = 0; i < B_LOADS; ++i)
      *reinterpret_cast<uint4*>(Bs + b_row[i] * 128 + ((chunk ^ (b_row[i] & 7)) << 4)) = rb[i];
  };

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int64_t KT = p.K / BK;
  load_slab(0);
  store_slab(0);
  __syncthreads();

  const int frow = lane & 31, fhalf = lane >> 5;
  for (int64_t kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < KT) load_slab((kt + 1) * BK);
    const char* As = smem + buf * STAGE;
    const char* Bs = As + BM * BK * 2;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int c = ks * 2 + fhalf;
      bf16x8_t af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int row = wm * TM + i * 32 + frow;
        af[i] = *reinterpret_cast<const bf16x8_t*>(As + row * 128 + ((c ^ (row & 7)) << 4));
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int row = wn * TN + j * 32 + frow;
        bfr[j] = *reinterpret_cast<const bf16x8_t*>(Bs + row * 128 + ((c ^ (row & 7)) << 4));
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < KT) store_slab(buf ^ 1);
    __syncthreads();
  }

  // acc[i][j][r] holds C[row, col] with col = lane % 32 and row = 8 (r / 4) + 4 (lane / 32) + r % 4.
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int64_t n = n0 + wn * TN + j * 32 + frow;
      if (n >= p.N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t m = m0 + wm * TM + i * 32 + 8 * (r >> 2) + 4 * fhalf + (r & 3);
        if (m < p.M) epi_store<true, EPI>(p, m, n, acc[i][j][r]);
      }
    }
}

// ------------------------------------------------------------------ float32
template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmParams p) {
  constexpr int T = 64, TK = 16;
  __shared__ float As[TK][T + 4];
  __shared__ float Ws[TK][T + 4];
  const int64_t m0 = static_cast<int64_t>(blockIdx.y) * T, n0 = static_cast<int64_t>(blockIdx.x) * T;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4] = {};
  const float* A1 = static_cast<const float*>(p.A1);
  const float* A2 = static_cast<const float*>(p.A2);
  const float* Wp = static_cast<const float*>(p.W);
  for (int64_t k0 = 0; k0 < p.K; k0 += TK) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = threadIdx.x + i * 256;  // 0..1023 over [64 rows][16 k]
      const int r = e >> 4, kk = e & 15;
      const int64_t k = k0 + kk;
      float av = 0.f, wv = 0.f;
      if (k < p.K) {
        const int64_t m = m0 + r, n = n0 + r;
        if (m < p.M) av = k < p.K1 ? A1[m * p.lda1 + k] : A2[m * p.lda2 + (k - p.K1)];
        if (n < p.N) wv = Wp[n * p.ldw + k];
      }
      As[kk][r] = av;
      Ws[kk][r] = wv;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) { a[i] = As[kk][ty * 4 + i]; b[i] = Ws[kk][tx * 4 + i]; }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t m = m0 + ty * 4 + i, n = n0 + tx * 4 + j;
      if (m < p.M && n < p.N) epi_store<false, EPI>(p, m, n, acc[i][j]);
    }
}

template <int BM, int BN, int WM, int WN, int EPI>
int launch_bf16(const GemmParams& p, hipStream_t s, const char* name, double flops, double bytes) {
  constexpr int smem = 2 * (BM + BN) * BK * 2;
  static bool attr_set = false;
  if (!attr_set) {
    FF_CHECK_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_bf16_kernel<BM, BN, WM, WN, EPI>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, smem),
                 "gemm smem attribute");
    attr_set = true;
  }
  const int64_t tiles = ((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN);
  LaunchScope ls(name, s, flops, bytes);
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WM, WN, EPI>), dim3(static_cast<unsigned>(tiles)),
                     dim3(WM * WN * 64), smem, s, p);
  return ls.status();
}

template <int EPI>
int dispatch_bf16(const GemmParams& p, hipStream_t s, double flops, double bytes) {
  static const char* names[3] = {"gemm_bf16", "gemm_bf16_gelu", "gemm_bf16_gated"};
  return launch_bf16<256, 256, 2, 4, EPI>(p, s, names[EPI], flops, bytes);
}

template <int EPI>
int dispatch_f32(const GemmParams& p, hipStream_t s, double flops, double bytes) {
  static const char* names[3] = {"gemm_f32", "gemm_f32_gelu", "gemm_f32_gated"};
  dim3 grid(static_cast<unsigned>((p.N + 63) / 64), static_cast<unsigned>((p.M + 63) / 64));
  LaunchScope ls(names[EPI], s, flops, bytes);
  hipLaunchKernelGGL(gemm_f32_kernel<EPI>, grid, dim3(256), 0, s, p);
  return ls.status();
}

}  // namespace

int gemm(const GemmArgs& a, hipStream_t s) {
  if (a.M == 0 || a.N == 0) return FF_OK;
  GemmParams p{a.M, a.N, a.K, a.A1, a.lda1, a.K1, a.A2 ? a.A2 : a.A1, a.A2 ? a.lda2 : a.lda1,
               a.W, a.ldw, a.bias, a.out, a.ldo, a.gelu_from, a.gate, a.gate_ld, a.resid, a.ldr,
               a.rows_per_sample > 0 ? a.rows_per_sample : a.M};
  const double esz = static_cast<double>(dtype_size(a.dtype));
  const double flops = 2.0 * a.M * a.N * a.K;
  const double bytes = esz * (static_cast<double>(a.M) * a.K + static_cast<double>(a.N) * a.K +
                              static_cast<double>(a.M) * a.N * (a.epi == EPI_GATED ? 2.0 : 1.0));
  if (a.dtype == FF_BF16) {
    if (a.K % BK != 0 || a.K1 % BK != 0)
      return fail(FF_EUNSUPPORTED, "gemm: bf16 K=%lld (K1=%lld) must be a multiple of %d", (long long)a.K,
                  (long long)a.K1, BK);
    switch (a.epi) {
      case EPI_NONE: return dispatch_bf16<EPI_NONE>(p, s, flops, bytes);
      case EPI_GELU: return dispatch_bf16<EPI_GELU>(p, s, flops, bytes);
      default: return dispatch_bf16<EPI_GATED>(p, s, flops, bytes);
    }
  }
  switch (a.epi) {
    case EPI_NONE: return dispatch_f32<EPI_NONE>(p, s, flops, bytes);
    case EPI_GELU: return dispatch_f32<EPI_GELU>(p, s, flops, bytes);
    default: return dispatch_f32<EPI_GATED>(p, s, flops, bytes);
  }
}

}  // namespace ff
