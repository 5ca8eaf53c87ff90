// Y = A W^T (+ epilogue) for the DiT's linear layers: QKV, output, MLP, embedders.
//
// bf16: MFMA 32x32x16 (gfx950) tiles, fp32 accumulation.  A [M, K] and W [N, K]
// are both K-contiguous (nn.Linear layout).  A workgroup computes a BM x BN
// tile; its waves split it into wave tiles, each a grid of 32x32 MFMA blocks.
// Large problems use a 256 x 256 tile computed by eight waves in a compute /
// memory ping-pong and fed by direct buffer->LDS loads of 64-wide K slabs
// (gemm_bf16_pp); small ones a 128 x 128 tile staged through registers with two
// LDS buffers (gemm_bf16_kernel).  gfx950's LDS serves a 16-byte-per-lane read
// for 16 lanes per clock across 64 banks (256 bytes), so LDS rows are stored
// with their 16-byte chunks permuted by a row-dependent XOR: the fragment reads
// of 16 consecutive rows land on 16 distinct bank groups.  Tiles are walked a
// few tile rows at a time so that tiles running together share A rows and W
// rows in L2.
//
// Epilogues fuse the bias, GELU-tanh (from a column on, for the fused
// single-stream projection), the adaLN-gated residual X + g * (.) and, on the
// QKV projections, the per-head QK norm, rotation and head-major relayout of
// the attention operands (epilogue_qkv).
//
// fp8: the same 256 x 256 ping-pong kernel on OCP E4M3 codes (gemm_fp8_pp):
// 128-wide K slabs (the same 128-byte LDS rows), the unscaled MFMA 32x32x64, and
// the per-row / per-column dequantisation scales applied in the epilogue before
// the bias.
//
// f32: a plain LDS-tiled FMA kernel with the same epilogues, for the float32
// configurations.
#include <type_traits>

#include "dev.h"
#include "ff_internal.h"

namespace ff {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef int i32x8_t __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) void lds_t;
typedef __attribute__((address_space(1))) void glb_t;

// EPI_QKV whose columns from 3H on are a single-stream block's MLP input (bias + GELU-tanh, stored
// to out): a kernel of its own, so the dual-stream QKV kernel carries no GELU code.
constexpr int EPI_QKV_GELU = 4;

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
  int64_t rows_per_sample;   // EPI_QKV: tokens per sample of the stream
  int vec_ok;   // 16-byte vector access of bias, gate, resid and out is aligned
  // EPI_QKV (fused): Q, K [B, heads, n_joint, 128] and V^T [B, heads, 128, n_joint] outputs, the
  // per-head RMSNorm weights, the (cos, sin) table [tokens, 64] (null: no rotation).
  bf16_t* q_out; bf16_t* k_out; bf16_t* vt_out;
  const bf16_t* q_w; const bf16_t* k_w; const float2* rope;
  int64_t hidden, n_joint, tok_offset, rope_from;
  int heads; float eps;
  // fp8: out = epi(row_scale[m] * col_scale[n] * acc + bias)
  const float* row_scale; const float* col_scale;
  // EPI_SUMSQ: row m's sum of squares of its stored columns [64 j, 64 j + 64), j < 2 sumsq_w / 64,
  // at sumsq[m * (2 sumsq_w / 64) + j]
  float* sumsq; int64_t sumsq_w;
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
template <int64_t GROUP_M = 8>
__device__ __forceinline__ void group_order(int64_t lid, int64_t num_m, int64_t num_n, int64_t& tm, int64_t& tn) {
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
//
// Split-K tail: when the tile count leaves a last round that fills only part of the GPU, the
// tiles from split_from on are each split into `parts` K ranges (work units split_from + S t + j,
// j = 0 .. S - 1).  Units j < S - 1 write their float32 partial sums to `partial` and publish them
// by storing `epoch` into their flag; unit S - 1, which is dispatched after them, waits for the
// flags, adds the partial sums and runs the epilogue.  split_from == tiles: no split.
struct GemmBatch {
  GemmParams p[2];
  int64_t tiles0, tiles;
  int64_t split_from;
  int parts;
  float4* partial;           // [split tiles][parts - 1][32 float4][512 threads]
  uint64_t* flags;           // [split tiles][parts - 1]
  uint64_t epoch;
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


// Epilogue of a wave's FM pairs of 32 x 64 accumulator blocks (the two column blocks of one
// block row; pair i at rows mw + 32 i, columns nw .. nw + 63).  Each pair goes through a per-wave
// 32 x 68 float scratch in LDS and comes back with lane l holding rows l / 8 + 8 q (q = 0..3),
// columns 8 (l % 8) .. + 7: every output row of a pair is one 128-byte line, written by 8 lanes
// with 16-byte non-temporal stores (the output streams to memory rather than through the caches:
// -5 to -8% on the write-bound epilogue).  A row stride of 68 floats keeps both the column writes
// and the 16-byte row reads free of bank conflicts.  Bias and gate (one row when the wave's rows
// lie in one sample) are loaded once, and each pair's residual rows are issued two pairs ahead,
// before the previous pair's stores, so no pair waits on the stores of another.
constexpr int PAIR_LD = 68;
__device__ __forceinline__ void transpose_blocks(const f32x16_t& a0, const f32x16_t& a1, float* scratch, int lane,
                                                 float (&v)[4][8]) {
  const int fcol = lane & 31, fhalf = lane >> 5;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int row = 8 * (r >> 2) + 4 * fhalf + (r & 3);
    scratch[row * PAIR_LD + fcol] = a0[r];
    scratch[row * PAIR_LD + 32 + fcol] = a1[r];
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  const int rr = lane >> 3, cc = (lane & 7) * 8;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 x = *reinterpret_cast<const float4*>(scratch + (rr + 8 * q) * PAIR_LD + cc);
    const float4 y = *reinterpret_cast<const float4*>(scratch + (rr + 8 * q) * PAIR_LD + cc + 4);
    v[q][0] = x.x; v[q][1] = x.y; v[q][2] = x.z; v[q][3] = x.w;
    v[q][4] = y.x; v[q][5] = y.y; v[q][6] = y.z; v[q][7] = y.w;
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}
template <int EPI, int FM, int FN, int JP, int I = 0>
__device__ __forceinline__ void transpose_pair(const f32x16_t (&acc)[FM][FN], float* scratch, int lane, float (&v)[4][8]) {
  transpose_blocks(acc[I][2 * JP], acc[I][2 * JP + 1], scratch, lane, v);
}

// Columns 64 JP .. 64 JP + 63 of the wave's FM x FN block grid (blocks 2 JP and 2 JP + 1 of each row).
template <int EPI, int FM, int FN = 2, int JP = 0, bool SCALED = false>
__device__ __forceinline__ void epilogue_pairs(const GemmParams& p, const f32x16_t (&acc)[FM][FN], int64_t mw, int64_t nw,
                                               float* scratch, int lane) {
  static_assert(FM <= 4, "pairs per wave");
  const int rr = lane >> 3, cc = (lane & 7) * 8;
  const int64_t n = nw + cc;
  bf16_t* out = static_cast<bf16_t*>(p.out);
  // Per lane: 16-byte vector path, or element-wise at a ragged right edge / unaligned operands.
  // The transposes below involve every lane, so they stay outside any per-lane branch.
  const bool vec = p.vec_ok && n + 8 <= p.N;
  float bv[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (vec && p.bias) ld8<true>(p.bias, n, bv);
  float cs[8];        // fp8: the lane's eight column scales
  if constexpr (SCALED) {
    if (vec) {
      const float4 c0 = *reinterpret_cast<const float4*>(p.col_scale + n);
      const float4 c1 = *reinterpret_cast<const float4*>(p.col_scale + n + 4);
      cs[0] = c0.x; cs[1] = c0.y; cs[2] = c0.z; cs[3] = c0.w; cs[4] = c1.x; cs[5] = c1.y; cs[6] = c1.z; cs[7] = c1.w;
    }
  }
  uint4 rs[2][4];     // residual rows of two pairs in flight (bf16)
  auto load_resid = [&](int i, uint4 (&dst)[4]) {
    if (!vec) return;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      int64_t m = mw + 32 * i + rr + 8 * q;
      if (m >= p.M) m = p.M - 1;
      dst[q] = *reinterpret_cast<const uint4*>(static_cast<const bf16_t*>(p.resid) + m * p.ldr + n);
    }
  };
  float gv[8];        // gate row of the wave's sample, when its rows lie in one sample
  bool one_sample = false;
  if constexpr (EPI == EPI_GATED) {
    load_resid(0, rs[0]);
    if (FM > 1) load_resid(1, rs[1]);
    const int64_t m_lo = mw < p.M ? mw : p.M - 1, m_hi = mw + 32 * FM - 1 < p.M ? mw + 32 * FM - 1 : p.M - 1;
    const uint64_t s_lo = static_cast<uint64_t>(m_lo) / static_cast<uint64_t>(p.rows_per_sample);
    one_sample = s_lo == static_cast<uint64_t>(m_hi) / static_cast<uint64_t>(p.rows_per_sample);
    if (vec && p.gate && one_sample) {
      const float4 g0 = *reinterpret_cast<const float4*>(p.gate + s_lo * p.gate_ld + n);
      const float4 g1 = *reinterpret_cast<const float4*>(p.gate + s_lo * p.gate_ld + n + 4);
      gv[0] = g0.x; gv[1] = g0.y; gv[2] = g0.z; gv[3] = g0.w;
      gv[4] = g1.x; gv[5] = g1.y; gv[6] = g1.z; gv[7] = g1.w;
    }
  }
  // EPI_SUMSQ: which 64-column slot of the row's partial sums this pair fills (-1: past 2 sumsq_w)
  const int64_t sq_slot = EPI == EPI_SUMSQ && nw < 2 * p.sumsq_w ? nw / 64 : -1;
  float v[4][8];
#define FF_PAIR(I)                                                                                   \
  if constexpr (I < FM) {                                                                            \
    transpose_pair<EPI, FM, FN, JP, I>(acc, scratch, lane, v);                                       \
    for (int q = 0; q < 4; ++q) {                                                                    \
      const int64_t m = mw + 32 * (I) + rr + 8 * q;                                                  \
      if (!vec) {                                                                                    \
        for (int e = 0; e < 8; ++e)                                                                  \
          if (m < p.M && n + e < p.N) {                                                              \
            float a = v[q][e];                                                                       \
            if constexpr (SCALED) a *= p.row_scale[m] * p.col_scale[n + e];                          \
            epi_store<true, EPI>(p, m, n + e, a);                                                    \
          }                                                                                          \
        continue;                                                                                    \
      }                                                                                              \
      float rsm = 1.f;                                                                               \
      if constexpr (SCALED) rsm = p.row_scale[m < p.M ? m : p.M - 1];                                \
      float g[8], r8[8];                                                                             \
      if constexpr (EPI == EPI_GATED) {                                                              \
        const uint32_t w[4] = {rs[(I) & 1][q].x, rs[(I) & 1][q].y, rs[(I) & 1][q].z, rs[(I) & 1][q].w};  \
        for (int j = 0; j < 4; ++j) {                                                                \
          r8[2 * j] = __uint_as_float(w[j] << 16);                                                   \
          r8[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);                                       \
        }                                                                                            \
        if (p.gate) {                                                                                \
          if (one_sample) {                                                                          \
            for (int e = 0; e < 8; ++e) g[e] = gv[e];                                                \
          } else {                                                                                   \
            const int64_t mc = m < p.M ? m : p.M - 1;                                                \
            const uint64_t smp = static_cast<uint64_t>(mc) / static_cast<uint64_t>(p.rows_per_sample); \
            for (int e = 0; e < 8; ++e) g[e] = p.gate[smp * p.gate_ld + n + e];                      \
          }                                                                                          \
        }                                                                                            \
      }                                                                                              \
      for (int e = 0; e < 8; ++e) {                                                                  \
        float x = v[q][e];                                                                           \
        if constexpr (SCALED) x *= rsm * cs[e];                                                      \
        x += bv[e];                                                                                  \
        if constexpr (EPI == EPI_GELU) {                                                             \
          if (n + e >= p.gelu_from) x = gelu_tanh_f(x);                                              \
        } else if constexpr (EPI == EPI_GATED) {                                                     \
          x = p.gate ? fmaf(g[e], x, r8[e]) : x + r8[e];                                             \
        }                                                                                            \
        v[q][e] = x;                                                                                 \
      }                                                                                              \
      if constexpr (EPI == EPI_SUMSQ) {                                                              \
        if (sq_slot >= 0) {                                                                          \
          float ss = 0.f;                                                                            \
          for (int e = 0; e < 8; ++e) {                                                              \
            const float r = bf2f(f2bf(v[q][e]));                                                     \
            ss = fmaf(r, r, ss);                                                                     \
          }                                                                                          \
          ss += __shfl_xor(ss, 1, 64);                                                               \
          ss += __shfl_xor(ss, 2, 64);                                                               \
          ss += __shfl_xor(ss, 4, 64);                                                               \
          if ((lane & 7) == 0 && m < p.M) p.sumsq[m * (2 * p.sumsq_w / 64) + sq_slot] = ss;          \
        }                                                                                            \
      }                                                                                              \
      if (m < p.M) st8_bf16_nt(out, m * p.ldo + n, v[q]);                                            \
    }                                                                                                \
    if constexpr (EPI == EPI_GATED && (I) + 2 < FM) load_resid((I) + 2, rs[(I) & 1]);                 \
  }
  FF_PAIR(0) FF_PAIR(1) FF_PAIR(2) FF_PAIR(3)
#undef FF_PAIR
}

// Fused QKV epilogue of a 64-token x 128-column wave tile, i.e. one head of Q, K or V for 64
// tokens of one stream (the QK norm and the rotation of the attention input, done while the
// projection is still in registers instead of by a second pass over the packed output).
//   Q, K: x = acc + bias; RMS over the head's 128 columns (a row's columns sit in 8 lanes of the
//         wave); y = x / rms * w; each column pair (2j, 2j + 1) of a token at or past rope_from
//         is rotated by (cos, sin) of pair j in table row token - rope_from (earlier tokens, the
//         text of a joint sequence, are not rotated); rows go to [B, heads, n_joint, 128] at
//         tok_offset + token.
//   V:    x = acc + bias, written transposed to [B, heads, 128, n_joint] through a per-wave
//         128 x 68 bf16 LDS scratch, so each head row leaves as 128 contiguous bytes.
// The norm is taken of the float32 projection (the two-pass path reads it back rounded to bf16).
constexpr int VT_LD = 68;   // bf16 row stride of the V^T scratch: conflict-free 8-byte writes
constexpr int QKV_SCRATCH = 128 * VT_LD * 2;   // bytes per wave (the Q/K transposes use less)
template <int FM, int FN>
__device__ __forceinline__ void epilogue_qkv(const GemmParams& p, const f32x16_t (&acc)[FM][FN], int64_t mw, int64_t nw,
                                             char* scratch, int lane) {
  static_assert(FM == 2 && FN == 4, "64 x 128 wave tile");
  const int part = static_cast<int>(nw / p.hidden);            // 0 Q, 1 K, 2 V (wave-uniform)
  const int64_t head = (nw % p.hidden) / 128;
  const int64_t S = p.rows_per_sample;
  const bf16_t* bias = static_cast<const bf16_t*>(p.bias);
  // Tokens of this wave: rows mw .. mw + 63 (clipped at M); one sample when they do not straddle.
  const int64_t m_last = mw + 63 < p.M ? mw + 63 : p.M - 1;
  const int64_t b_lo = mw / S;
  const bool one_sample = b_lo == m_last / S;
  if (part < 2) {
    const int rr = lane >> 3, cc = (lane & 7) * 8;
    bf16_t* dst = part == 0 ? p.q_out : p.k_out;
    const bf16_t* wn = part == 0 ? p.q_w : p.k_w;
    float bv[2][8], wv[2][8];
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      if (bias) {
        ld8<true>(bias, nw + 64 * h2 + cc, bv[h2]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) bv[h2][e] = 0.f;
      }
      ld8<true>(wn, 64 * h2 + cc, wv[h2]);
    }
    float* fs = reinterpret_cast<float*>(scratch);
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      float v[2][4][8];
      transpose_blocks(acc[i][0], acc[i][1], fs, lane, v[0]);
      transpose_blocks(acc[i][2], acc[i][3], fs, lane, v[1]);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t m = mw + 32 * i + rr + 8 * q;
        float ss = 0.f;
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            v[h2][q][e] += bv[h2][e];
            ss = fmaf(v[h2][q][e], v[h2][q][e], ss);
          }
        ss += __shfl_xor(ss, 1, 64);
        ss += __shfl_xor(ss, 2, 64);
        ss += __shfl_xor(ss, 4, 64);
        const float rstd = rsqrtf(ss * (1.0f / 128.0f) + p.eps);
        const int64_t mc = m < p.M ? m : p.M - 1;
        const int64_t b = one_sample ? b_lo : mc / S;
        const int64_t tok = mc - b * S;
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
          float cs[8];
          if (p.rope && tok >= p.rope_from) {
            const float4* rp = reinterpret_cast<const float4*>(p.rope + (tok - p.rope_from) * 64 + 32 * h2 + cc / 2);
            const float4 r0 = rp[0], r1 = rp[1];
            cs[0] = r0.x; cs[1] = r0.y; cs[2] = r0.z; cs[3] = r0.w; cs[4] = r1.x; cs[5] = r1.y; cs[6] = r1.z; cs[7] = r1.w;
          } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) { cs[2 * j] = 1.f; cs[2 * j + 1] = 0.f; }
          }
          float y[8];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float x0 = v[h2][q][2 * j] * rstd * wv[h2][2 * j], x1 = v[h2][q][2 * j + 1] * rstd * wv[h2][2 * j + 1];
            y[2 * j] = x0 * cs[2 * j] - x1 * cs[2 * j + 1];
            y[2 * j + 1] = x0 * cs[2 * j + 1] + x1 * cs[2 * j];
          }
          if (m < p.M) st8<true>(dst, ((b * p.heads + head) * p.n_joint + p.tok_offset + tok) * 128 + 64 * h2 + cc, y);
        }
      }
    }
    return;
  }
  // V: [token][d] accumulators -> [d][token] bf16 scratch -> 128-byte rows of V^T.
  bf16_t* vs = reinterpret_cast<bf16_t*>(scratch);
  const int fcol = lane & 31, fhalf = lane >> 5;
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    const float bj = bias ? bf2f(bias[nw + 32 * j + fcol]) : 0.f;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        uint2 w;
        w.x = uint32_t(f2bf(acc[i][j][4 * g4] + bj)) | (uint32_t(f2bf(acc[i][j][4 * g4 + 1] + bj)) << 16);
        w.y = uint32_t(f2bf(acc[i][j][4 * g4 + 2] + bj)) | (uint32_t(f2bf(acc[i][j][4 * g4 + 3] + bj)) << 16);
        *reinterpret_cast<uint2*>(vs + (32 * j + fcol) * VT_LD + 32 * i + 8 * g4 + 4 * fhalf) = w;
      }
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  const int c8 = lane & 7;
  bf16_t* vt = p.vt_out;
  const bool whole = one_sample && mw + 64 <= p.M;
  const int64_t tok0 = mw - b_lo * S;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int d = k * 8 + (lane >> 3);
    const uint4 w = *reinterpret_cast<const uint4*>(vs + d * VT_LD + 8 * c8);
    if (whole) {
      *reinterpret_cast<uint4*>(vt + ((b_lo * p.heads + head) * 128 + d) * p.n_joint + p.tok_offset + tok0 + 8 * c8) = w;
    } else {
      const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int64_t m = mw + 8 * c8 + e;
        if (m >= p.M) continue;
        const int64_t b = m / S, tok = m - b * S;
        vt[((b * p.heads + head) * 128 + d) * p.n_joint + p.tok_offset + tok] =
            static_cast<bf16_t>(e & 1 ? ws[e >> 1] >> 16 : ws[e >> 1] & 0xffffu);
      }
    }
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

// ------------------------------------------------------------------ bf16, 256 x 256, ping-pong
// Eight waves, two per SIMD, in two groups of four (wave w and wave w + 4 share a SIMD).
// Each wave owns a 128 x 64 block of the 256 x 256 tile (4 x 2 MFMA blocks) and alternates
// between a compute phase (the 32 MFMAs of one 64-wide K slab) and a memory phase (the LDS
// reads of the fragments it needs next); the groups are one phase apart, so one wave of a
// SIMD keeps the matrix core busy while the other feeds itself.  A barrier separates
// phases: slab s is computed by group 0 in phase 2s and by group 1 in phase 2s + 1, so it
// is read from LDS in phases 2s - 1 and 2s only and two 64 KB buffers suffice.  Slab
// s + 2's direct loads go into slab s's buffer during phase 2s + 1 (both groups are done
// with it): group 0 issues the A rows in its memory phase, group 1 the W rows between the
// first MFMAs of its compute phase, and each waits for its own loads one phase later, before
// the barrier that publishes the slab.  Loads go through buffer resources whose record count
// ends at the matrix's last row, so rows past M (or N) read as zero without a per-row
// clamp; K rows are 128-byte lines (a 64-wide slab), stored with the chunk swizzle
// chunk ^ ((row >> 1) & 7).

__device__ __forceinline__ u32x4_t buffer_rsrc(const void* base, uint64_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  u32x4_t r;
  r.x = static_cast<uint32_t>(a);
  r.y = static_cast<uint32_t>(a >> 32);   // stride 0: raw buffer, range check on the offset
  r.z = static_cast<uint32_t>(bytes < 0xffffffffull ? bytes : 0xffffffffull);
  r.w = 0x00020000u;                      // 32-bit data format
  return r;
}
// One 16-byte-per-lane direct load from a buffer into LDS at the wave-uniform `lds` address.
// Written as inline assembly: the compiler's wait-count pass cannot tell an LDS-DMA
// destination from the fragment reads and would wait for every load before any LDS read;
// the kernel orders them itself (vmcnt wait + barrier before a slab is read).
// The statement writes M0, a register the compiler reserves (hence clang's -Winline-asm note on
// the clobber).  Nothing in these kernels keeps a compiler value in M0 across it: the compiler
// uses M0 only for its own LDS-DMA builtins, s_sendmsg, lane reads with an SGPR index and
// relative moves, and none of them occur here; the clobber keeps the declaration honest.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma_buf16(const u32x4_t& rsrc, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :: "s"(lds), "v"(voff), "s"(rsrc) : "memory", "m0");
}
#pragma clang diagnostic pop

// For outputs whose tile columns come in whole sixteens: within each group of 16 tile rows, runs
// of 256 launch slots cover a 16 x 16 block of tiles, and the 32 slots of one XCD (consecutive
// slots go to consecutive XCDs) a 4 x 8 part of it, so the tiles an XCD runs at once share 4 A and
// 8 W panels in its L2 instead of 2 and 16.  Measured 2% faster than the plain walk on the
// 12288-wide MLP-up output and 2% slower on 3072- and 9216-wide ones, which keep the plain walk.
__device__ __forceinline__ void xcd_block_order(int64_t lid, int64_t num_m, int64_t num_n, int64_t& tm, int64_t& tn) {
  const int64_t in_group = 16 * num_n;
  const int64_t first_m = lid / in_group * 16;
  if (num_m - first_m < 16) {
    group_order<16>(lid, num_m, num_n, tm, tn);
    return;
  }
  const int64_t r = lid % in_group, st = r >> 8, q = r & 255, x = q & 7, j = q >> 3;
  tm = first_m + 4 * (x & 3) + (j & 3);
  tn = 16 * st + 8 * (x >> 2) + (j >> 2);
}

// LAYOUT 0: each wave a 128 x 64 block (wm = w4 / 2, wn = 2 grp + w4 % 2); LAYOUT 1: a 64 x 128
// block (wm = w4, wn = grp), one whole 128-column head, for the fused QKV epilogue.  The two
// waves of a SIMD (same w4) always share their A rows.  F8: operands are E4M3 codes; a slab is
// 128 of them, read as two k64 steps of 32 bytes per lane (lane half h takes bytes 32 h ..
// 32 h + 31 of the step, for A and W alike) into the unscaled MFMA 32x32x64.
template <int EPI, int LAYOUT, bool F8>
__device__ __forceinline__ void pp_body(const GemmBatch& batch) {
  constexpr int ES = F8 ? 1 : 2;                              // bytes per element
  constexpr int BM = 256, BN = 256, ROWB = 128, KS = ROWB / ES;   // 128-byte LDS rows
  constexpr int STAGE = (BM + BN) * ROWB;                     // 64 KB
  constexpr int KSTEPS = F8 ? 2 : 4;                          // MFMA k steps per slab
  static_assert(!F8 || (EPI == EPI_NONE || EPI == EPI_GELU), "fp8 epilogues: bias, GELU");
  constexpr int TM = LAYOUT == 0 ? 128 : 64, TN = LAYOUT == 0 ? 64 : 128;
  constexpr int FM = TM / 32, FN = TN / 32;
  static_assert((EPI != EPI_QKV && EPI != EPI_QKV_GELU) || LAYOUT == 1, "the fused QKV epilogue needs a head per wave");
  constexpr int A_INS = BM / 8 / 4, B_INS = BN / 8 / 4;       // 1 KB loads per wave per slab
  extern __shared__ __attribute__((aligned(16))) char smem[];

  // Plain launch order (consecutive tiles on different XCDs) walking 16 tile rows at a time:
  // measured faster than giving each XCD a contiguous range, or 4, 8 or 32 rows, on the DiT's
  // shapes; XCD blocks where the tile columns come in sixteens.
  const int64_t unit = blockIdx.x;
  int part = 0, parts = 1;
  int64_t lid = unit;
  if (unit >= batch.split_from) {
    parts = batch.parts;
    lid = batch.split_from + (unit - batch.split_from) / parts;
    part = static_cast<int>((unit - batch.split_from) % parts);
  }
  const int which = lid >= batch.tiles0 ? 1 : 0;
  const GemmParams& p = batch.p[which];
  const int64_t num_m = (p.M + BM - 1) / BM, num_n = (p.N + BN - 1) / BN;
  int64_t tm, tn;
  if (num_n % 16 == 0)
    xcd_block_order(lid - (which ? batch.tiles0 : 0), num_m, num_n, tm, tn);
  else
    group_order<16>(lid - (which ? batch.tiles0 : 0), num_m, num_n, tm, tn);
  const int64_t m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 2, w4 = wave & 3;
  const int wm = LAYOUT == 0 ? w4 >> 1 : w4, wn = LAYOUT == 0 ? grp * 2 + (w4 & 1) : grp;
  // This unit's slabs: [s_begin, s_begin + KT) of the tile's p.K / KS (all of them when unsplit).
  const int KT_all = static_cast<int>(p.K / KS), KT1 = static_cast<int>(p.K1 / KS);
  const int s_begin = part * KT_all / parts;
  const int KT = (part + 1) * KT_all / parts - s_begin;

  // Load q of a wave fills LDS rows 32 q + 8 w4 .. + 7 of its matrix; lane l lands at
  // row + l / 8, stored chunk l % 8, so it fetches logical chunk (l % 8) ^ ((row >> 1) & 7),
  // which does not depend on q.
  const int lrow = 8 * w4 + (lane >> 3);
  const int lck = (lane & 7) ^ ((lrow >> 1) & 7);
  const int64_t rows_a = p.M - m0, rows_b = p.N - n0;
  // A may come from two sources (the two-part K of the fused single-stream projection):
  // slabs [0, KT1) from A1, the rest from A2.
  const bool two = KT1 > 0 && KT1 < KT_all;
  const char* a1_tile = static_cast<const char*>(p.A1) + m0 * p.lda1 * ES;
  const char* a2_tile = static_cast<const char*>(p.A2) + m0 * p.lda2 * ES;
  const int64_t a1_bytes = rows_a * p.lda1 * ES, a2_bytes = rows_a * p.lda2 * ES;
  const uint32_t a1_off = static_cast<uint32_t>(lrow * p.lda1 * ES + lck * 16);
  const uint32_t a2_off = static_cast<uint32_t>(lrow * p.lda2 * ES + lck * 16);
  const uint32_t a1_step = static_cast<uint32_t>(32 * p.lda1 * ES), a2_step = static_cast<uint32_t>(32 * p.lda2 * ES);
  const char* b_tile = static_cast<const char*>(p.W) + n0 * p.ldw * ES;
  const int64_t b_bytes = rows_b * p.ldw * ES;
  const uint32_t b_off = static_cast<uint32_t>(lrow * p.ldw * ES + lck * 16);
  const uint32_t b_step = static_cast<uint32_t>(32 * p.ldw * ES);
  const uint32_t smem_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(smem));
  auto rsrc_b = [&](int s) {   // s counts this unit's slabs
    const int64_t db = static_cast<int64_t>(s_begin + s) * ROWB;
    return buffer_rsrc(b_tile + db, static_cast<uint64_t>(b_bytes - db));
  };
  auto issue_a = [&](int s, int dst) {   // this unit's slab s's A rows into the buffer of its slab dst
    const int sa = s_begin + s;
    const bool second = two && sa >= KT1;
    const int64_t da = static_cast<int64_t>(second ? sa - KT1 : sa) * ROWB;
    const u32x4_t r = buffer_rsrc((second ? a2_tile : a1_tile) + da, static_cast<uint64_t>((second ? a2_bytes : a1_bytes) - da));
    const uint32_t off = second ? a2_off : a1_off, step = second ? a2_step : a1_step;
    const uint32_t lds = smem_base + (dst & 1) * STAGE + w4 * 1024;
#pragma unroll
    for (int q = 0; q < A_INS; ++q) dma_buf16(r, off + q * step, lds + q * 4096);
  };

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
  // One slab of fragments, [k step][block]: 16 bytes per lane (bf16, k16 steps) or 32 (fp8, k64).
  typedef typename std::conditional<F8, i32x8_t, bf16x8_t>::type frag_t;
  frag_t fa[KSTEPS][FM], fb[KSTEPS][FN];
  auto read_frags = [&](int s) {
    const char* S = smem + (s & 1) * STAGE;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      if constexpr (F8) {
        const int c0 = ((ks * 4 + fhalf * 2) ^ key) << 4, c1 = ((ks * 4 + fhalf * 2 + 1) ^ key) << 4;
        auto rd32 = [&](int off) {
          const u32x4_t lo = *reinterpret_cast<const u32x4_t*>(S + off + c0);
          const u32x4_t hi = *reinterpret_cast<const u32x4_t*>(S + off + c1);
          return i32x8_t{int(lo.x), int(lo.y), int(lo.z), int(lo.w), int(hi.x), int(hi.y), int(hi.z), int(hi.w)};
        };
#pragma unroll
        for (int i = 0; i < FM; ++i) fa[ks][i] = rd32(a_frag0 + i * 32 * ROWB);
#pragma unroll
        for (int j = 0; j < FN; ++j) fb[ks][j] = rd32(b_frag0 + j * 32 * ROWB);
      } else {
        const int coff = ((ks * 2 + fhalf) ^ key) << 4;
#pragma unroll
        for (int i = 0; i < FM; ++i) fa[ks][i] = *reinterpret_cast<const bf16x8_t*>(S + a_frag0 + i * 32 * ROWB + coff);
#pragma unroll
        for (int j = 0; j < FN; ++j) fb[ks][j] = *reinterpret_cast<const bf16x8_t*>(S + b_frag0 + j * 32 * ROWB + coff);
      }
    }
  };
  // The MFMAs of a slab (32 bf16 or 16 fp8); with `rb` set, the eight W-row loads of a later
  // slab go out one after each of the first eight MFMAs: the loads must land by the end of the
  // next phase, and issuing them early in this one gives them most of two phases to arrive
  // (spread evenly over the phase, the last one had little more than one).
  auto compute = [&](const u32x4_t* rb, uint32_t lds_b) {
    static_assert(KSTEPS * FM * FN >= 8, "eight loads per compute phase");
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          if constexpr (F8)   // zero scale operands: the compiler emits the unscaled v_mfma_f32_32x32x64_f8f6f4
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fa[ks][i], fb[ks][j], acc[i][j], 0, 0, 0, 0, 0, 0);
          else
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[ks][i], fb[ks][j], acc[i][j], 0, 0, 0);
          const int idx = (ks * FM + i) * FN + j;
          if (rb != nullptr && idx < 8) {
            const int q = idx;
            dma_buf16(*rb, b_off + q * b_step, lds_b + q * 4096);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
  };

  // Two code paths, one per group (the group is wave-uniform), with the same number of
  // barriers; a single loop branching on the group would keep both groups' fragments live at
  // once.  The last two slabs are peeled: no loads are issued past the end of K, and after the
  // barrier that ends phase 2 KT - 2 nothing reads the LDS ring any more, so group 0 starts its
  // epilogue while group 1 computes the last slab (each wave's scratch is its own).
  if (grp == 0) {
    issue_a(0, 0);
    if (KT > 1) {
      issue_a(1, 1);
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(A_INS) : "memory");   // A of slab 0 has landed
    } else {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    wg_barrier();
    read_frags(0);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    wg_barrier();
    for (int s = 0; s + 2 < KT; ++s) {
      compute(nullptr, 0);                                 // phase 2s
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");    // A of slab s + 1 has landed
      wg_barrier();
      read_frags(s + 1);                                   // phase 2s + 1
      issue_a(s + 2, s);
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      wg_barrier();
    }
    if (KT > 1) {                                          // slab KT - 2
      compute(nullptr, 0);
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      wg_barrier();
      read_frags(KT - 1);
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      wg_barrier();
    }
    compute(nullptr, 0);                                   // slab KT - 1
    __builtin_amdgcn_sched_barrier(0);
    wg_barrier();
  } else {
    {
      const uint32_t lds = smem_base + w4 * 1024 + BM * ROWB;
      const u32x4_t r0 = rsrc_b(0);
#pragma unroll
      for (int q = 0; q < B_INS; ++q) dma_buf16(r0, b_off + q * b_step, lds + q * 4096);
      if (KT > 1) {
        const u32x4_t r1 = rsrc_b(1);
#pragma unroll
        for (int q = 0; q < B_INS; ++q) dma_buf16(r1, b_off + q * b_step, lds + STAGE + q * 4096);
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(B_INS) : "memory");   // W of slab 0 has landed
      } else {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      }
    }
    wg_barrier();
    wg_barrier();
    for (int s = 0; s + 2 < KT; ++s) {
      read_frags(s);                                       // phase 2s
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");    // W of slab s + 1 has landed
      wg_barrier();
      const u32x4_t rb = rsrc_b(s + 2);                   // phase 2s + 1
      compute(&rb, smem_base + (s & 1) * STAGE + w4 * 1024 + BM * ROWB);
      __builtin_amdgcn_sched_barrier(0);
      wg_barrier();
    }
    if (KT > 1) {                                          // slab KT - 2
      read_frags(KT - 2);
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      wg_barrier();
      compute(nullptr, 0);
      __builtin_amdgcn_sched_barrier(0);
      wg_barrier();
    }
    read_frags(KT - 1);                                    // slab KT - 1
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    wg_barrier();
    compute(nullptr, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (parts > 1) {
    // Split tile: float4 q of thread tid's accumulators is (block q / 4 of the wave's FM x FN grid,
    // elements 4 (q % 4) ..); partial block b holds it at [q][tid], so each store and load of a
    // wave covers 1 KB contiguously.
    constexpr int NQ = FM * FN * 4;
    const int64_t st = lid - batch.split_from;
    uint64_t* flag = batch.flags + st * (parts - 1);
    float4* blocks = batch.partial + st * (parts - 1) * (NQ * 512);
    if (part < parts - 1) {
      float4* dst = blocks + static_cast<int64_t>(part) * (NQ * 512) + tid;
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const f32x16_t& a = acc[(q >> 2) / FN][(q >> 2) % FN];
        dst[q * 512] = make_float4(a[4 * (q & 3)], a[4 * (q & 3) + 1], a[4 * (q & 3) + 2], a[4 * (q & 3) + 3]);
      }
      // Every thread's stores have reached the XCD's L2; one release by thread 0 then writes the L2
      // back and publishes the flag (a fence per wave would write it back eight times).
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      if (tid == 0) __hip_atomic_store(flag + part, batch.epoch, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
      return;
    }
    // The last part: wait for the others (they have lower unit ids, so they were dispatched
    // first; the spin is bounded so a wave always finishes), then add their sums in part order.
    // The polls are relaxed loads (an acquire per poll would invalidate the XCD's L2 under the
    // tiles still computing there); one acquire after the last poll orders the partial loads.
    if (tid < parts - 1) {
      for (int spin = 0; spin < (1 << 22); ++spin) {
        if (__hip_atomic_load(flag + tid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == batch.epoch) break;
        __builtin_amdgcn_s_sleep(2);
      }
    }
    if (tid < 64) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    __syncthreads();
    for (int j = 0; j < parts - 1; ++j) {
      const float4* src = blocks + static_cast<int64_t>(j) * (NQ * 512) + tid;
      // four loads in flight at a time: all of them at once would not fit beside the accumulators
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const float4 v = src[q * 512];
        f32x16_t& a = acc[(q >> 2) / FN][(q >> 2) % FN];
        a[4 * (q & 3)] += v.x;
        a[4 * (q & 3) + 1] += v.y;
        a[4 * (q & 3) + 2] += v.z;
        a[4 * (q & 3) + 3] += v.w;
        if ((q & 3) == 3) __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  if constexpr (EPI == EPI_QKV) {
    epilogue_qkv<FM, FN>(p, acc, m0 + wm * TM, n0 + wn * TN, smem + wave * QKV_SCRATCH, lane);
  } else if constexpr (EPI == EPI_QKV_GELU) {
    // A wave's 128 columns are all Q/K/V (below 3H) or all MLP input: 3H is a multiple of 128.
    const int64_t mw = m0 + wm * TM, nw = n0 + wn * TN;
    if (nw < 3 * p.hidden) {
      epilogue_qkv<FM, FN>(p, acc, mw, nw, smem + wave * QKV_SCRATCH, lane);
    } else {
      float* fs = reinterpret_cast<float*>(smem + wave * QKV_SCRATCH);
      epilogue_pairs<EPI_GELU, FM, FN, 0>(p, acc, mw, nw, fs, lane);
      epilogue_pairs<EPI_GELU, FM, FN, 1>(p, acc, mw, nw + 64, fs, lane);
    }
  } else {
    static_assert(FN == 2 && 8 * 32 * PAIR_LD * 4 <= 2 * STAGE, "epilogue scratch fits the LDS ring");
    epilogue_pairs<EPI, FM, FN, 0, F8>(p, acc, m0 + wm * TM, n0 + wn * TN,
                                       reinterpret_cast<float*>(smem) + wave * 32 * PAIR_LD, lane);
  }
}

template <int EPI, int LAYOUT>
__global__ __launch_bounds__(512, 1) void gemm_bf16_pp(GemmBatch batch) {
  pp_body<EPI, LAYOUT, false>(batch);
}
template <int EPI>
__global__ __launch_bounds__(512, 1) void gemm_fp8_pp(GemmBatch batch) {
  pp_body<EPI, 0, true>(batch);
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
  static std::atomic<uint64_t> limit_set{0};
  FF_TRY(ensure_smem_limit(reinterpret_cast<const void*>(&gemm_bf16_kernel<BM, BN, WM, WN, EPI>), smem, limit_set));
  const int64_t tiles = ((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN);
  LaunchScope ls(name, s, flops, bytes);
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WM, WN, EPI>), dim3(static_cast<unsigned>(tiles)),
                     dim3(WM * WN * 64), smem, s, p);
  return ls.status();
}

// Compute units of the current device (one 256 x 256 tile runs per CU at a time).
int device_cus(int* out) {
  static std::atomic<int> cus[64] = {};
  int dev = 0;
  FF_CHECK_HIP(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(FF_EUNSUPPORTED, "device ordinal %d above 63", dev);
  int n = cus[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    FF_CHECK_HIP(hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev), "CU count");
    cus[dev].store(n, std::memory_order_relaxed);
  }
  *out = n;
  return FF_OK;
}

// Split-K plan of a launch: the tiles of a last, partly filled round are split into S K ranges
// so that the round's work units fill the CUs, S = min(CUs / tail, slabs / 8, 8), when the
// workspace holds the partial sums, both problems have the same number of slabs and K has at
// least 96 slabs.  Measured on the DiT's shapes with 1632 tiles (6.375 rounds): the K = 12288
// projection gains 3.5%; at K = 3072 half a tile is too short for the fixup (partial sums through
// memory, an L2 write-back) to pay, and those launches were 0-1.5% slower, so they are not split.
constexpr int kSplitMinSlabs = 8, kSplitMaxParts = 8, kSplitMinK = 96;
constexpr size_t kSplitBlockBytes = 512 * 128 * 4;   // one tile's partial sums (512 threads x 128 floats)
std::atomic<uint64_t> g_split_epoch{0x5EED000000000000ull};

void plan_split(GemmBatch& b, int cus, void* ws, size_t ws_bytes, int slab_k) {
  b.split_from = b.tiles;
  b.parts = 1;
  const int64_t tail = cus > 0 ? b.tiles % cus : 0;
  if (!ws || tail == 0 || b.p[0].K != b.p[1].K || b.tiles < cus) return;
  const int64_t slabs = b.p[0].K / slab_k;
  if (slabs < kSplitMinK) return;
  int64_t S = cus / tail;
  if (S > slabs / kSplitMinSlabs) S = slabs / kSplitMinSlabs;
  if (S > kSplitMaxParts) S = kSplitMaxParts;
  if (S < 2) return;
  const size_t n_blocks = static_cast<size_t>(tail) * (S - 1);
  const size_t flag_bytes = round_up(n_blocks * sizeof(uint64_t), 256);
  if (flag_bytes + n_blocks * kSplitBlockBytes > ws_bytes) return;
  b.split_from = b.tiles - tail;
  b.parts = static_cast<int>(S);
  b.flags = static_cast<uint64_t*>(ws);
  b.partial = reinterpret_cast<float4*>(static_cast<char*>(ws) + flag_bytes);
  b.epoch = g_split_epoch.fetch_add(1, std::memory_order_relaxed) + 1;
}

int64_t split_units(const GemmBatch& b) { return b.split_from + (b.tiles - b.split_from) * b.parts; }

template <int EPI>
int launch_pp_batch(const GemmBatch& b0, hipStream_t s, const char* name, double flops, double bytes, void* ws = nullptr,
                    size_t ws_bytes = 0) {
  constexpr bool qkv = EPI == EPI_QKV || EPI == EPI_QKV_GELU;
  constexpr int LAYOUT = qkv ? 1 : 0;
  constexpr int ring = 2 * 512 * 64 * 2;
  constexpr int smem = qkv && 8 * QKV_SCRATCH > ring ? 8 * QKV_SCRATCH : ring;
  static std::atomic<uint64_t> limit_set{0};
  FF_TRY(ensure_smem_limit(reinterpret_cast<const void*>(&gemm_bf16_pp<EPI, LAYOUT>), smem, limit_set));
  GemmBatch b = b0;
  int cus = 0;
  FF_TRY(device_cus(&cus));
  plan_split(b, cus, ws, ws_bytes, BK);
  LaunchScope ls(name, s, flops, bytes);
  hipLaunchKernelGGL((gemm_bf16_pp<EPI, LAYOUT>), dim3(static_cast<unsigned>(split_units(b))), dim3(512), smem, s, b);
  return ls.status();
}

int64_t tiles256(const GemmParams& p) { return ((p.M + 255) / 256) * ((p.N + 255) / 256); }

template <int EPI>
int launch_fp8(const GemmParams& p, hipStream_t s, const char* name, double flops, double bytes) {
  constexpr int smem = 2 * 512 * 128;
  static std::atomic<uint64_t> limit_set{0};
  FF_TRY(ensure_smem_limit(reinterpret_cast<const void*>(&gemm_fp8_pp<EPI>), smem, limit_set));
  GemmBatch b{};
  b.p[0] = p;
  b.p[1] = p;
  b.tiles0 = b.tiles = tiles256(p);
  b.split_from = b.tiles;   // no split-K
  b.parts = 1;
  LaunchScope ls(name, s, flops, bytes);
  hipLaunchKernelGGL((gemm_fp8_pp<EPI>), dim3(static_cast<unsigned>(b.tiles)), dim3(512), smem, s, b);
  return ls.status();
}

const char* const kGemmNames[5] = {"gemm_bf16", "gemm_bf16_gelu", "gemm_bf16_gated", "gemm_bf16_qkv",
                                   "gemm_bf16_qkv_gelu"};

// Problems with at least one 256 x 256 tile per CU take the 256 x 256 kernel;
// smaller ones the 128 x 128 tile, which fills more CUs.
template <int EPI>
int dispatch_bf16(const GemmParams& p, hipStream_t s, double flops, double bytes, void* ws, size_t ws_bytes) {
  if (tiles256(p) >= 256) {
    GemmBatch b{};
    b.p[0] = p;
    b.p[1] = p;
    b.tiles0 = b.tiles = tiles256(p);
    return launch_pp_batch<EPI>(b, s, kGemmNames[EPI], flops, bytes, ws, ws_bytes);
  }
  return launch_bf16<128, 128, 2, 2, EPI>(p, s, kGemmNames[EPI], flops, bytes);
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
  if (a.qkv) {
    const QkvArgs& q = *a.qkv;
    p.q_out = static_cast<bf16_t*>(q.Q); p.k_out = static_cast<bf16_t*>(q.Kd); p.vt_out = static_cast<bf16_t*>(q.Vt);
    p.q_w = static_cast<const bf16_t*>(q.q_w); p.k_w = static_cast<const bf16_t*>(q.k_w); p.rope = q.rope;
    p.hidden = static_cast<int64_t>(q.heads) * 128; p.n_joint = q.n_joint; p.tok_offset = q.tok_offset;
    p.rope_from = q.rope_from;
    p.heads = q.heads; p.eps = q.eps;
    p.rows_per_sample = q.src_rows;
  }
  p.sumsq = a.sumsq;
  p.sumsq_w = a.sumsq_w;
  return p;
}

}  // namespace

bool gemm_sumsq_ok(const GemmArgs& a) {
  return a.dtype == FF_BF16 && a.K % BK == 0 && a.K1 == a.K && a.N % 64 == 0 && a.ldo % 8 == 0 && aligned16(a.out) &&
         (!a.bias || aligned16(a.bias)) && a.sumsq && a.sumsq_w > 0 && a.sumsq_w % 64 == 0 && 2 * a.sumsq_w <= a.N &&
         ((a.M + 255) / 256) * ((a.N + 255) / 256) >= 256;
}

namespace {

// The QKV projection of one stream can end in the fused norm / rotation / relayout epilogue:
// bf16, 128-wide heads with a per-head norm, every GEMM row a token (rows = B x tokens), V taken
// transposed, and the 16-byte alignment and 8-token granularity the vector stores need.
bool qkv_fusable(const GemmArgs& a) {
  if (!a.qkv || a.dtype != FF_BF16) return false;
  const QkvArgs& q = *a.qkv;
  const int64_t H = static_cast<int64_t>(q.heads) * 128;
  return q.dtype == FF_BF16 && q.d == 128 && !q.full_width_norm && q.apply_norm && q.v_transposed &&
         (a.N == 3 * H || (a.N > 3 * H && a.gelu_from == 3 * H)) && a.K1 == a.K && q.src_rows == q.n_tok && a.M == q.B * q.n_tok && q.n_tok % 8 == 0 &&
         q.n_joint % 8 == 0 && q.tok_offset % 8 == 0 && aligned16(q.Q) && aligned16(q.Kd) && aligned16(q.Vt) &&
         aligned16(q.q_w) && aligned16(q.k_w) && (!q.rope || aligned16(q.rope)) && (!a.bias || aligned16(a.bias));
}
double gemm_flops(const GemmArgs& a) { return 2.0 * a.M * a.N * a.K; }
double gemm_bytes(const GemmArgs& a) {
  const double esz = static_cast<double>(dtype_size(a.dtype));
  return esz * (static_cast<double>(a.M) * a.K + static_cast<double>(a.N) * a.K +
                static_cast<double>(a.M) * a.N * (a.epi == EPI_GATED ? 2.0 : 1.0));
}
}  // namespace

size_t gemm_split_bytes() {
  constexpr size_t max_blocks = 255;   // tail x (S - 1) < 256 CUs
  return round_up(max_blocks * sizeof(uint64_t), 256) + max_blocks * kSplitBlockBytes;
}

int gemm(const GemmArgs& a, hipStream_t s) {
  if (a.M == 0 || a.N == 0) return FF_OK;
  if (a.epi == EPI_QKV) {
    GemmParams p = make_params(a);
    const bool tail = a.qkv && a.N > 3 * static_cast<int64_t>(a.qkv->heads) * a.qkv->d;   // MLP columns
    if (qkv_fusable(a) && a.K % BK == 0 && tiles256(p) >= 256) {
      GemmBatch b{};
      b.p[0] = p;
      b.p[1] = p;
      b.tiles0 = b.tiles = tiles256(p);
      if (tail)
        return launch_pp_batch<EPI_QKV_GELU>(b, s, kGemmNames[EPI_QKV_GELU], gemm_flops(a), gemm_bytes(a), a.split_ws,
                                             a.split_bytes);
      return launch_pp_batch<EPI_QKV>(b, s, kGemmNames[EPI_QKV], gemm_flops(a), gemm_bytes(a), a.split_ws,
                                      a.split_bytes);
    }
    GemmArgs plain = a;   // two passes: the packed projection, then the norm / rotation / relayout
    plain.epi = tail ? EPI_GELU : EPI_NONE;
    plain.qkv = nullptr;
    FF_TRY(gemm(plain, s));
    return a.qkv ? qk_norm_rope(*a.qkv, s) : fail(FF_EINVAL, "gemm: QKV epilogue without its arguments");
  }
  GemmParams p = make_params(a);
  const double flops = gemm_flops(a), bytes = gemm_bytes(a);
  if (a.epi == EPI_SUMSQ) {
    if (!gemm_sumsq_ok(a)) return fail(FF_EUNSUPPORTED, "gemm: the sum-of-squares epilogue does not apply to this shape");
    GemmBatch b{};
    b.p[0] = p;
    b.p[1] = p;
    b.tiles0 = b.tiles = tiles256(p);
    return launch_pp_batch<EPI_SUMSQ>(b, s, kGemmNames[EPI_NONE], flops, bytes, a.split_ws, a.split_bytes);
  }
  if (a.dtype == FF_BF16) {
    if (a.K % BK != 0 || a.K1 % BK != 0)
      return fail(FF_EUNSUPPORTED, "gemm: bf16 K=%lld (K1=%lld) must be a multiple of %d", (long long)a.K,
                  (long long)a.K1, BK);
    switch (a.epi) {
      case EPI_NONE: return dispatch_bf16<EPI_NONE>(p, s, flops, bytes, a.split_ws, a.split_bytes);
      case EPI_GELU: return dispatch_bf16<EPI_GELU>(p, s, flops, bytes, a.split_ws, a.split_bytes);
      default: return dispatch_bf16<EPI_GATED>(p, s, flops, bytes, a.split_ws, a.split_bytes);
    }
  }
  switch (a.epi) {
    case EPI_NONE: return dispatch_f32<EPI_NONE>(p, s, flops, bytes);
    case EPI_GELU: return dispatch_f32<EPI_GELU>(p, s, flops, bytes);
    default: return dispatch_f32<EPI_GATED>(p, s, flops, bytes);
  }
}

int gemm_fp8(const Fp8GemmArgs& a, hipStream_t s) {
  if (a.M == 0 || a.N == 0) return FF_OK;
  if (a.K % 128 != 0) return fail(FF_EUNSUPPORTED, "gemm_fp8: K=%lld must be a multiple of 128", (long long)a.K);
  GemmParams p{};
  p.M = a.M; p.N = a.N; p.K = a.K;
  p.A1 = a.A; p.lda1 = a.lda; p.K1 = a.K; p.A2 = a.A; p.lda2 = a.lda;
  p.W = a.W; p.ldw = a.ldw; p.bias = a.bias;
  p.out = a.out; p.ldo = a.ldo; p.gelu_from = a.gelu_from;
  p.rows_per_sample = a.M;
  p.row_scale = a.d_a; p.col_scale = a.d_w;
  p.vec_ok = a.ldo % 8 == 0 && aligned16(a.out) && (!a.bias || aligned16(a.bias)) && aligned16(a.d_w);
  const double flops = 2.0 * a.M * a.N * a.K;
  const double bytes = static_cast<double>(a.M) * a.K + static_cast<double>(a.N) * a.K + 2.0 * a.M * a.N +
                       4.0 * (a.M + a.N);
  if (a.epi == EPI_GELU) return launch_fp8<EPI_GELU>(p, s, "gemm_fp8_gelu", flops, bytes);
  return launch_fp8<EPI_NONE>(p, s, "gemm_fp8", flops, bytes);
}

int gemm2(const GemmArgs& a0, const GemmArgs& a1, hipStream_t s) {
  if (a0.epi == EPI_QKV || a1.epi == EPI_QKV) {
    const bool tail0 = a0.qkv && a0.N > 3 * static_cast<int64_t>(a0.qkv->heads) * a0.qkv->d;
    const bool tail1 = a1.qkv && a1.N > 3 * static_cast<int64_t>(a1.qkv->heads) * a1.qkv->d;
    if (tail0 || tail1 || a0.epi != a1.epi) {   // only two plain QKV projections are grouped
      FF_TRY(gemm(a0, s));
      return gemm(a1, s);
    }
    GemmBatch b{};
    b.p[0] = make_params(a0);
    b.p[1] = make_params(a1);
    b.tiles0 = tiles256(b.p[0]);
    b.tiles = b.tiles0 + tiles256(b.p[1]);
    if (a0.epi == EPI_QKV && a1.epi == EPI_QKV && qkv_fusable(a0) && qkv_fusable(a1) && a0.K % BK == 0 &&
        a1.K % BK == 0 && b.tiles >= 256)
      return launch_pp_batch<EPI_QKV>(b, s, kGemmNames[EPI_QKV], gemm_flops(a0) + gemm_flops(a1),
                                      gemm_bytes(a0) + gemm_bytes(a1), a0.split_ws, a0.split_bytes);
    GemmArgs p0 = a0, p1 = a1;   // two passes for both streams
    if (p0.epi == EPI_QKV) { p0.epi = EPI_NONE; p0.qkv = nullptr; }
    if (p1.epi == EPI_QKV) { p1.epi = EPI_NONE; p1.qkv = nullptr; }
    FF_TRY(gemm2(p0, p1, s));
    if (a0.epi == EPI_QKV) FF_TRY(a0.qkv ? qk_norm_rope(*a0.qkv, s) : fail(FF_EINVAL, "gemm2: QKV epilogue without its arguments"));
    if (a1.epi == EPI_QKV) FF_TRY(a1.qkv ? qk_norm_rope(*a1.qkv, s) : fail(FF_EINVAL, "gemm2: QKV epilogue without its arguments"));
    return FF_OK;
  }
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
  switch (a0.epi) {
    case EPI_NONE: return launch_pp_batch<EPI_NONE>(b, s, kGemmNames[EPI_NONE], flops, bytes, a0.split_ws, a0.split_bytes);
    case EPI_GELU: return launch_pp_batch<EPI_GELU>(b, s, kGemmNames[EPI_GELU], flops, bytes, a0.split_ws, a0.split_bytes);
    default: return launch_pp_batch<EPI_GATED>(b, s, kGemmNames[EPI_GATED], flops, bytes, a0.split_ws, a0.split_bytes);
  }
}

}  // namespace ff
