// Y = A W^T (+ epilogue) for the DiT's linear layers: QKV, output, MLP, embedders.
//
// bf16: MFMA 32x32x16 (gfx950) tiles, fp32 accumulation.  A [M, K] and W [N, K]
// are both K-contiguous (nn.Linear layout).  A workgroup computes a BM x BN
// tile; its waves split it into wave tiles, each a grid of 32x32 MFMA blocks.
// Large problems use a 256 x 256 tile with one wave per SIMD fed by direct
// global->LDS loads of 64-wide K slabs (gemm_bf16_256); small ones a 128 x 128
// tile staged through registers with two LDS buffers (gemm_bf16_kernel).  gfx950's LDS serves a
// 16-byte-per-lane read for 16 lanes per clock across 64 banks (256 bytes), so
// LDS rows are stored with their 16-byte chunks permuted by a row-dependent
// XOR: the fragment reads of 16 consecutive rows land on 16 distinct bank
// groups.  Tiles are ordered so that consecutive tiles of one XCD (workgroups
// are dealt round-robin over the 8 XCDs) share A rows in that XCD's L2.
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
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_t;
typedef __attribute__((address_space(1))) void glb_t;

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
  int vec_ok;   // 16-byte vector access of bias, gate, resid and out is aligned
};

template <bool BF16, int EPI>
__device__ __forceinline__ void epi_store(const GemmParams& p, int64_t m, int64_t n, float acc) {
  float v = acc;
  if (p.bias) v += ld1<BF16>(p.bias, n);
  if constexpr (EPI == EPI_GELU) {
    if (n >= p.gelu_from) v = gelu_tanh_f(v);
  } else if constexpr (EPI == EPI_GATED) {
    const float g = p.gate ? p.gate[(m / p.rows_per_sample) * p.gate_ld + n] : 1.0f;
    v = ld1<BF16>(p.resid, m * p.ldr + n) + g * v;
  }
  st1<BF16>(p.out, m * p.ldo + n, v);
}

// Maps the linear workgroup id to a (tile_m, tile_n) pair: first regroup ids
// so each XCD owns a contiguous range, then walk GROUP_M tile rows at a time.
__device__ __forceinline__ int64_t xcd_remap(int64_t pid, int64_t total) {
  const int64_t full = total / 8 * 8;
  return pid < full ? (pid % 8) * (full / 8) + pid / 8 : pid;
}
__device__ __forceinline__ void group_order(int64_t lid, int64_t num_m, int64_t num_n, int64_t& tm, int64_t& tn) {
  constexpr int64_t GROUP_M = 8;
  const int64_t in_group = GROUP_M * num_n;
  const int64_t gidx = lid / in_group;
  const int64_t first_m = gidx * GROUP_M;
  const int64_t gsize = (num_m - first_m) < GROUP_M ? (num_m - first_m) : GROUP_M;
  const int64_t r = lid % in_group;
  tm = first_m + r % gsize;
  tn = r / gsize;
}
__device__ __forceinline__ void tile_coords(int64_t pid, int64_t num_m, int64_t num_n, int64_t& tm,
                                            int64_t& tn) {
  group_order(xcd_remap(pid, num_m * num_n), num_m, num_n, tm, tn);
}

// Up to two GEMM problems with the same tile kernel in one launch (the text and
// image streams of a dual-stream block): tiles [0, tiles0) belong to p[0].
struct GemmBatch {
  GemmParams p[2];
  int64_t tiles0, tiles;
};

constexpr int BK = 64;

// Epilogue of one wave's FM x FN grid of 32x32 accumulator blocks.  Each block
// goes through a per-wave 32 x 36 float scratch in LDS (the K loop is over, so
// LDS is free) and comes back row-major: lane l owns row l/2, 16 consecutive
// columns, so bias, gate and residual are read and the output written with
// 16-byte vector accesses, one sample-index division per row.
template <int EPI>
__device__ __forceinline__ void epilogue_block(const GemmParams& p, const f32x16_t& a, int64_t mb, int64_t nb,
                                               float* scratch, int lane) {
  const int frow = lane & 31, fhalf = lane >> 5;
  const int rr = lane >> 1, cc = (lane & 1) * 16;
  const bf16_t* bias = static_cast<const bf16_t*>(p.bias);
  bf16_t* out = static_cast<bf16_t*>(p.out);
#pragma unroll
  for (int r = 0; r < 16; ++r) scratch[(8 * (r >> 2) + 4 * fhalf + (r & 3)) * 36 + frow] = a[r];
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  float v[16];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 t = *reinterpret_cast<const float4*>(scratch + rr * 36 + cc + 4 * q);
    v[4 * q] = t.x; v[4 * q + 1] = t.y; v[4 * q + 2] = t.z; v[4 * q + 3] = t.w;
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  const int64_t m = mb + rr;
  const int64_t n = nb + cc;
  if (m >= p.M || n >= p.N) return;
  if (p.vec_ok && n + 16 <= p.N) {
    if (bias) {
      float b[16];
      ld8<true>(bias, n, *reinterpret_cast<float(*)[8]>(b));
      ld8<true>(bias, n + 8, *reinterpret_cast<float(*)[8]>(b + 8));
#pragma unroll
      for (int e = 0; e < 16; ++e) v[e] += b[e];
    }
    if constexpr (EPI == EPI_GELU) {
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (n + e >= p.gelu_from) v[e] = gelu_tanh_f(v[e]);
    } else if constexpr (EPI == EPI_GATED) {
      float rs[16];
      ld8<true>(p.resid, m * p.ldr + n, *reinterpret_cast<float(*)[8]>(rs));
      ld8<true>(p.resid, m * p.ldr + n + 8, *reinterpret_cast<float(*)[8]>(rs + 8));
      if (p.gate) {
        const uint64_t smp = static_cast<uint64_t>(m) / static_cast<uint64_t>(p.rows_per_sample);
        const float* g = p.gate + smp * p.gate_ld + n;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float4 t = *reinterpret_cast<const float4*>(g + 4 * q);
          v[4 * q] = fmaf(t.x, v[4 * q], rs[4 * q]);
          v[4 * q + 1] = fmaf(t.y, v[4 * q + 1], rs[4 * q + 1]);
          v[4 * q + 2] = fmaf(t.z, v[4 * q + 2], rs[4 * q + 2]);
          v[4 * q + 3] = fmaf(t.w, v[4 * q + 3], rs[4 * q + 3]);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) v[e] += rs[e];
      }
    }
    st8<true>(out, m * p.ldo + n, *reinterpret_cast<const float(*)[8]>(v));
    st8<true>(out, m * p.ldo + n + 8, *reinterpret_cast<const float(*)[8]>(v + 8));
  } else {
#pragma unroll
    for (int e = 0; e < 16; ++e)
      if (n + e < p.N) epi_store<true, EPI>(p, m, n + e, v[e]);
  }
}

// All FM x FN blocks of a wave, block (i, j) at rows mw + 32 i, columns nw + 32 j.  The
// recursion keeps every accumulator index a compile-time constant (a dynamic index would
// send the whole accumulator array to scratch memory).
template <int EPI, int FM, int FN, int B = 0>
__device__ __forceinline__ void epilogue_blocks(const GemmParams& p, const f32x16_t (&acc)[FM][FN], int64_t mw,
                                                int64_t nw, float* scratch, int lane) {
  if constexpr (B < FM * FN) {
    epilogue_block<EPI>(p, acc[B / FN][B % FN], mw + (B / FN) * 32, nw + (B % FN) * 32, scratch, lane);
    epilogue_blocks<EPI, FM, FN, B + 1>(p, acc, mw, nw, scratch, lane);
  }
}


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

  // Global loads of this thread: row (tid + i*THREADS)/8, 16-byte chunk tid%8, staged
  // through registers and written to LDS at chunk ^ ((row >> 1) & 7).  Rows past the
  // matrix edge are clamped.
  const int chunk = tid & 7;
  const bf16_t* a_src[A_LOADS];
  const bf16_t* b_src[B_LOADS];
  int a_lds[A_LOADS], b_lds[B_LOADS];
#pragma unroll
  for (int i = 0; i < A_LOADS; ++i) {
    const int row = (tid + i * THREADS) >> 3;
    const int64_t g = m0 + row < p.M ? m0 + row : p.M - 1;
    a_src[i] = static_cast<const bf16_t*>(p.A1) + g * p.lda1 + chunk * 8;
    a_lds[i] = row * 128 + ((chunk ^ ((row >> 1) & 7)) << 4);
  }
#pragma unroll
  for (int i = 0; i < B_LOADS; ++i) {
    const int row = (tid + i * THREADS) >> 3;
    const int64_t g = n0 + row < p.N ? n0 + row : p.N - 1;
    b_src[i] = static_cast<const bf16_t*>(p.W) + g * p.ldw + chunk * 8;
    b_lds[i] = BM * BK * 2 + row * 128 + ((chunk ^ ((row >> 1) & 7)) << 4);
  }

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int frow = lane & 31, fhalf = lane >> 5;
  // LDS byte offsets of this lane's fragment rows (chunk 0), and the row's swizzle key.
  int a_frag[FM], b_frag[FN];
#pragma unroll
  for (int i = 0; i < FM; ++i) a_frag[i] = (wm * TM + i * 32 + frow) * 128;
#pragma unroll
  for (int j = 0; j < FN; ++j) b_frag[j] = BM * BK * 2 + (wn * TN + j * 32 + frow) * 128;
  const int key = (frow >> 1) & 7;   // the same for every fragment row of this lane

  const int64_t KT = p.K / BK;
  const int64_t KT1 = p.K1 / BK;   // slab at which A switches to the second source
  u32x4_t ra[A_LOADS], rb[B_LOADS];

  // Issue the global loads of the current source pointers into registers, then
  // (after the current slab's MFMAs) write them to stage `buf`.
#define FF_GEMM_ISSUE()                                                                            \
  _Pragma("unroll") for (int i = 0; i < A_LOADS; ++i) ra[i] = *reinterpret_cast<const u32x4_t*>(a_src[i]); \
  _Pragma("unroll") for (int i = 0; i < B_LOADS; ++i) rb[i] = *reinterpret_cast<const u32x4_t*>(b_src[i]);
#define FF_GEMM_COMMIT(buf)                                                                        \
  {                                                                                                \
    char* D_ = smem + (buf) * STAGE;                                                               \
    _Pragma("unroll") for (int i = 0; i < A_LOADS; ++i) *reinterpret_cast<u32x4_t*>(D_ + a_lds[i]) = ra[i]; \
    _Pragma("unroll") for (int i = 0; i < B_LOADS; ++i) *reinterpret_cast<u32x4_t*>(D_ + b_lds[i]) = rb[i]; \
  }

  FF_GEMM_ISSUE()
  FF_GEMM_COMMIT(0)
  __syncthreads();

  for (int64_t kt = 0; kt < KT; ++kt) {
    const int buf = static_cast<int>(kt & 1);
    const bool more = kt + 1 < KT;
    if (more) {
      if (kt + 1 == KT1) {
        // continue K in the second A source
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i) {
          const int row = (tid + i * THREADS) >> 3;
          const int64_t g = m0 + row < p.M ? m0 + row : p.M - 1;
          a_src[i] = static_cast<const bf16_t*>(p.A2) + g * p.lda2 + chunk * 8;
        }
      } else {
#pragma unroll
        for (int i = 0; i < A_LOADS; ++i) a_src[i] += BK;
      }
#pragma unroll
      for (int i = 0; i < B_LOADS; ++i) b_src[i] += BK;
      FF_GEMM_ISSUE()
    }
    const char* S = smem + buf * STAGE;
    // Fragments of k16 step ks + 1 are read while the MFMAs of step ks run.
    bf16x8_t af[2][FM], bfr[2][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) af[0][i] = *reinterpret_cast<const bf16x8_t*>(S + a_frag[i] + ((fhalf ^ key) << 4));
#pragma unroll
    for (int j = 0; j < FN; ++j) bfr[0][j] = *reinterpret_cast<const bf16x8_t*>(S + b_frag[j] + ((fhalf ^ key) << 4));
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int cur = ks & 1;
      if (ks + 1 < BK / 16) {
        const int coff = (((ks + 1) * 2 + fhalf) ^ key) << 4;
#pragma unroll
        for (int i = 0; i < FM; ++i) af[cur ^ 1][i] = *reinterpret_cast<const bf16x8_t*>(S + a_frag[i] + coff);
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[cur ^ 1][j] = *reinterpret_cast<const bf16x8_t*>(S + b_frag[j] + coff);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      FF_GEMM_COMMIT(buf ^ 1)
    }
    __syncthreads();
  }
#undef FF_GEMM_ISSUE
#undef FF_GEMM_COMMIT

  // acc[i][j][r] holds C[row, col] with col = lane % 32 and row = 8 (r / 4) + 4 (lane / 32) + r % 4.
  __syncthreads();
  epilogue_blocks<EPI, FM, FN>(p, acc, m0 + wm * TM, n0 + wn * TN,
                               reinterpret_cast<float*>(smem) + wave * 32 * 36, lane);
}

// Workgroup barrier that no instruction (memory or not) is scheduled across.
__device__ __forceinline__ void wg_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// ------------------------------------------------------------------ bf16, 256 x 256 tiles
// 256 x 256 tile, one wave per SIMD, each wave a 128 x 128 grid of 4 x 4 MFMA
// blocks.  K advances in slabs of 64, so every row segment a direct load
// fetches is a whole 128-byte cache line (32-wide slabs fetch half lines, which
// halves the L2 -> LDS rate); two 64 KB LDS buffers.  Half a slab (two k16
// steps) of fragments sits in each of two register sets: the second half of
// slab s is read from LDS while the first half's MFMAs run, and the first half
// of slab s + 1 while the second half's run.  Per slab: barrier X (everyone has
// read slab s) lets slab s + 2's loads go into slab s's buffer between the
// MFMAs of the third k16 step; barrier Y (each wave has waited for its own
// loads of slab s + 1) publishes slab s + 1.  Loads past the end of K replay
// the last slab, so the number in flight is the same on every step.
template <int EPI>
__global__ __launch_bounds__(256, 1) void gemm_bf16_256(GemmBatch batch) {
  constexpr int BM = 256, BN = 256, WAVES = 4;
  constexpr int KS = 64, ROWB = KS * 2, CPR = ROWB / 16, RPI = 1024 / ROWB;   // 128-byte rows, 8 rows per load
  constexpr int TM = 128, TN = 128, FM = 4, FN = 4;
  constexpr int A_INS = BM / RPI / WAVES, B_INS = BN / RPI / WAVES, LPW = A_INS + B_INS;   // 8 + 8
  constexpr int STAGE = (BM + BN) * ROWB;   // 64 KB
  extern __shared__ __attribute__((aligned(16))) char smem[];

  const int64_t lid = xcd_remap(blockIdx.x, batch.tiles);
  const int which = lid >= batch.tiles0 ? 1 : 0;
  const GemmParams& p = batch.p[which];
  const int64_t num_m = (p.M + BM - 1) / BM, num_n = (p.N + BN - 1) / BN;
  int64_t tm, tn;
  group_order(lid - (which ? batch.tiles0 : 0), num_m, num_n, tm, tn);
  const int64_t m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // Load i of this wave fills rows RPI (i*WAVES + wave) .. +RPI-1 (1 KB of LDS); lane l lands at
  // row + l/CPR, stored chunk l%CPR, so it fetches logical chunk (l%CPR) ^ ((row >> 1) & 7).
  // Sources: a uniform base (the tile's first row) plus 32-bit per-lane byte offsets.
  const char* a_base = reinterpret_cast<const char*>(static_cast<const bf16_t*>(p.A1) + m0 * p.lda1);
  const char* b_base = reinterpret_cast<const char*>(static_cast<const bf16_t*>(p.W) + n0 * p.ldw);
  uint32_t a_off[A_INS], b_off[B_INS];
  auto a_offsets = [&](int64_t lda) {
#pragma unroll
    for (int i = 0; i < A_INS; ++i) {
      const int row = (i * WAVES + wave) * RPI + lane / CPR;
      const int ck = (lane % CPR) ^ ((row >> 1) & 7);
      const int64_t r = m0 + row < p.M ? row : p.M - 1 - m0;
      a_off[i] = static_cast<uint32_t>((r * lda + ck * 8) * 2);
    }
  };
  a_offsets(p.lda1);
#pragma unroll
  for (int i = 0; i < B_INS; ++i) {
    const int row = (i * WAVES + wave) * RPI + lane / CPR;
    const int ck = (lane % CPR) ^ ((row >> 1) & 7);
    const int64_t r = n0 + row < p.N ? row : p.N - 1 - n0;
    b_off[i] = static_cast<uint32_t>((r * p.ldw + ck * 8) * 2);
  }
  const int KT = static_cast<int>(p.K / KS), KT1 = static_cast<int>(p.K1 / KS);

  auto switch_a = [&](int slab) {
    if (slab == KT1 && slab > 0 && slab < KT) {
      // continue K in the second A source (the two-source single-stream projection)
      a_base = reinterpret_cast<const char*>(static_cast<const bf16_t*>(p.A2) + m0 * p.lda2);
      a_offsets(p.lda2);
    }
  };
  // Loads [first, first + count) of slab `slab` (A loads, then B loads).
  auto issue_part = [&](int slab, int first, int count) {
    const uint32_t back = slab < KT ? 0u : static_cast<uint32_t>(KS * 2);
    char* base = smem + (slab & 1) * STAGE + wave * 1024;
#pragma unroll
    for (int q = first; q < first + count; ++q) {
      if (q < A_INS) {
        __builtin_amdgcn_global_load_lds((const glb_t*)(a_base + (a_off[q] - back)), (lds_t*)(base + q * WAVES * 1024), 16, 0, 0);
        a_off[q] += KS * 2 - back;
      } else {
        const int i = q - A_INS;
        __builtin_amdgcn_global_load_lds((const glb_t*)(b_base + (b_off[i] - back)), (lds_t*)(base + BM * ROWB + i * WAVES * 1024), 16, 0, 0);
        b_off[i] += KS * 2 - back;
      }
    }
  };
  auto issue = [&](int slab) { issue_part(slab, 0, LPW); };

  f32x16_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int frow = lane & 31, fhalf = lane >> 5;
  const int key = (frow >> 1) & 7;
  const int a_frag0 = (wm * TM + frow) * ROWB, b_frag0 = BM * ROWB + (wn * TN + frow) * ROWB;
  // Register sets: r0 = k16 steps 0, 1 of a slab; r1 = steps 2, 3.  [step][block]
  bf16x8_t ra0[2][FM], rb0[2][FN], ra1[2][FM], rb1[2][FN];
  auto read_half = [&](int slab, int half, bf16x8_t (&ra)[2][FM], bf16x8_t (&rb)[2][FN]) {
    const char* S = smem + (slab & 1) * STAGE;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int coff = (((half * 2 + ks) * 2 + fhalf) ^ key) << 4;
#pragma unroll
      for (int i = 0; i < FM; ++i) ra[ks][i] = *reinterpret_cast<const bf16x8_t*>(S + a_frag0 + i * 32 * ROWB + coff);
#pragma unroll
      for (int j = 0; j < FN; ++j) rb[ks][j] = *reinterpret_cast<const bf16x8_t*>(S + b_frag0 + j * 32 * ROWB + coff);
    }
  };
  auto mfma_step = [&](const bf16x8_t (&ra)[FM], const bf16x8_t (&rb)[FN]) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ra[i], rb[j], acc[i][j], 0, 0, 0);
  };

  switch_a(0);
  issue(0);
  switch_a(1);
  issue(1);
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LPW) : "memory");   // slab 0 has landed
  wg_barrier();
  read_half(0, 0, ra0, rb0);
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  // Loads of slab s + 2 per k16 step 1, 2, 3 (the address unit takes a 1 KB load every
  // 16 clocks, so the 64 loads of a slab are spread over three steps of MFMAs).
  constexpr int G1 = 6, G2 = 5, G3 = LPW - G1 - G2;
  for (int s = 0; s < KT; ++s) {
    // step 0: read steps 2, 3 of slab s between the MFMAs
    read_half(s, 1, ra1, rb1);
    mfma_step(ra0[0], rb0[0]);
#pragma unroll
    for (int m = 0; m < FM * FN; ++m) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    switch_a(s + 2);
    wg_barrier();                                     // X: every wave has read slab s
    // steps 1, 2: slab s + 2's first loads into slab s's buffer
    issue_part(s + 2, 0, G1 + G2);
    mfma_step(ra0[1], rb0[1]);
    mfma_step(ra1[0], rb1[0]);
#pragma unroll
    for (int m = 0; m < 2 * FM * FN; ++m) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (m < FM * FN ? m < G1 : m - FM * FN < G2) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(G1 + G2) : "memory");   // slab s + 1 has landed
    wg_barrier();                                     // Y: publish slab s + 1
    // step 3: the rest of the loads; read steps 0, 1 of slab s + 1 (past the end: replayed data)
    issue_part(s + 2, G1 + G2, G3);
    read_half(s + 1, 0, ra0, rb0);
    mfma_step(ra1[1], rb1[1]);
#pragma unroll
    for (int m = 0; m < FM * FN; ++m) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      if (m < G3) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }

  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // replayed loads may still target LDS
  __syncthreads();
  epilogue_blocks<EPI, FM, FN>(p, acc, m0 + wm * TM, n0 + wn * TN,
                               reinterpret_cast<float*>(smem) + wave * 32 * 36, lane);
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
int launch_256_batch(const GemmBatch& b, hipStream_t s, const char* name, double flops, double bytes) {
  constexpr int smem = 2 * 512 * 64 * 2;
  static bool attr_set = false;
  if (!attr_set) {
    FF_CHECK_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_bf16_256<EPI>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, smem),
                 "gemm smem attribute");
    attr_set = true;
  }
  LaunchScope ls(name, s, flops, bytes);
  hipLaunchKernelGGL((gemm_bf16_256<EPI>), dim3(static_cast<unsigned>(b.tiles)), dim3(256), smem, s, b);
  return ls.status();
}

int64_t tiles256(const GemmParams& p) { return ((p.M + 255) / 256) * ((p.N + 255) / 256); }

// Problems with at least one 256 x 256 tile per CU take the 256 x 256 kernel;
// smaller ones the 128 x 128 tile, which fills more CUs.
template <int EPI>
int dispatch_bf16(const GemmParams& p, hipStream_t s, double flops, double bytes) {
  static const char* names[3] = {"gemm_bf16", "gemm_bf16_gelu", "gemm_bf16_gated"};
  if (tiles256(p) >= 256) {
    GemmBatch b{};
    b.p[0] = p;
    b.p[1] = p;
    b.tiles0 = b.tiles = tiles256(p);
    return launch_256_batch<EPI>(b, s, names[EPI], flops, bytes);
  }
  return launch_bf16<128, 128, 2, 2, EPI>(p, s, names[EPI], flops, bytes);
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

namespace {
GemmParams make_params(const GemmArgs& a) {
  GemmParams p{a.M, a.N, a.K, a.A1, a.lda1, a.K1, a.A2 ? a.A2 : a.A1, a.A2 ? a.lda2 : a.lda1,
               a.W, a.ldw, a.bias, a.out, a.ldo, a.gelu_from, a.gate, a.gate_ld, a.resid, a.ldr,
               a.rows_per_sample > 0 ? a.rows_per_sample : a.M, 0};
  p.vec_ok = a.ldo % 8 == 0 && aligned16(a.out) && (!a.bias || aligned16(a.bias)) &&
             (a.epi != EPI_GATED || (a.ldr % 8 == 0 && aligned16(a.resid) && (!a.gate || (a.gate_ld % 4 == 0 && aligned16(a.gate)))));
  return p;
}
double gemm_flops(const GemmArgs& a) { return 2.0 * a.M * a.N * a.K; }
double gemm_bytes(const GemmArgs& a) {
  const double esz = static_cast<double>(dtype_size(a.dtype));
  return esz * (static_cast<double>(a.M) * a.K + static_cast<double>(a.N) * a.K +
                static_cast<double>(a.M) * a.N * (a.epi == EPI_GATED ? 2.0 : 1.0));
}
}  // namespace

int gemm(const GemmArgs& a, hipStream_t s) {
  if (a.M == 0 || a.N == 0) return FF_OK;
  GemmParams p = make_params(a);
  const double flops = gemm_flops(a), bytes = gemm_bytes(a);
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

int gemm2(const GemmArgs& a0, const GemmArgs& a1, hipStream_t s) {
  const bool grouped = a0.dtype == FF_BF16 && a1.dtype == FF_BF16 && a0.epi == a1.epi && a0.M > 0 && a1.M > 0 &&
                       a0.N > 0 && a1.N > 0 && a0.K % BK == 0 && a1.K % BK == 0 && a0.K1 % BK == 0 &&
                       a1.K1 % BK == 0;
  if (!grouped) {
    FF_TRY(gemm(a0, s));
    return gemm(a1, s);
  }
  GemmBatch b{};
  b.p[0] = make_params(a0);
  b.p[1] = make_params(a1);
  b.tiles0 = tiles256(b.p[0]);
  b.tiles = b.tiles0 + tiles256(b.p[1]);
  if (b.tiles < 256) {
    FF_TRY(gemm(a0, s));
    return gemm(a1, s);
  }
  const double flops = gemm_flops(a0) + gemm_flops(a1), bytes = gemm_bytes(a0) + gemm_bytes(a1);
  static const char* names[3] = {"gemm_bf16", "gemm_bf16_gelu", "gemm_bf16_gated"};
  switch (a0.epi) {
    case EPI_NONE: return launch_256_batch<EPI_NONE>(b, s, names[0], flops, bytes);
    case EPI_GELU: return launch_256_batch<EPI_GELU>(b, s, names[1], flops, bytes);
    default: return launch_256_batch<EPI_GATED>(b, s, names[2], flops, bytes);
  }
}

}  // namespace ff
