// Joint (text + image) attention O = softmax(Q K^T / sqrt(d)) V, non-causal.
//
// bf16, d = 128: a flash-style kernel with online softmax in float32.  Each
// wave owns 32 queries; a workgroup of WAVES waves shares 64-key tiles of K
// and V^T staged through a ring of LDS buffers by direct global->LDS loads.
// Both products are computed
// transposed on MFMA 32x32x16:
//   S^T (keys x queries) = K Q^T        A = K rows (LDS), B = Q (registers)
//   O^T (d x queries)   += V^T P^T      A = V^T rows (LDS), B = P (registers)
// so a lane always holds one query (lane % 32): the running max, the running
// sum and the rescale of O are lane-local, and the only cross-lane step per
// tile is one exchange of the row max between the two lane halves.
// K rows are fed to the first MFMA in an order that swaps bits 2 and 3 of the
// row index; with it, the 8 scores a lane holds for a 16-key slice are keys
// 16s + 8(lane/32) + 0..7 in order, exactly the B-operand slots of the second
// MFMA, so P goes from accumulators to operands without any shuffle.
//
// float32 (any d <= 64): one thread per query with the same online softmax,
// for the small float32 configuration.
#include <cmath>

#include "dev.h"
#include "ff_internal.h"

namespace ff {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

struct AttnParams {
  int64_t B, heads, n_q, n_kv;
  const bf16_t* Q; const bf16_t* K; const bf16_t* Vt;
  bf16_t* out0; bf16_t* out1; int64_t split; int64_t ldo;
  float scale_log2;
  int64_t q_bs, q_hs, q_rs;   // Q element (b, h, q, :) at b*q_bs + h*q_hs + q*q_rs
};

constexpr int D = 128;
constexpr int KT = 64;                   // keys per tile
constexpr int K_STAGE = KT * D * 2;      // bytes of one K tile (64 rows x 256 B)
constexpr int V_STAGE = D * KT * 2;      // bytes of one V^T tile (128 rows x 128 B)

// LDS layouts.  gfx950's LDS serves 16-byte-per-lane reads for 16 lanes per
// clock over 64 banks (256 bytes); the chunk swizzles below put the fragment
// rows read by 16 consecutive lanes on 16 distinct bank groups.
// 16-byte chunk c of K row r (16 chunks per 256-byte row).
__device__ __forceinline__ int k_off(int r, int c) { return r * 256 + ((c ^ (r & 15)) << 4); }
// 16-byte chunk c of V^T row r (8 chunks per 128-byte row).
__device__ __forceinline__ int v_off(int r, int c) { return r * 128 + ((c ^ ((r >> 1) & 7)) << 4); }

typedef __attribute__((address_space(3))) void lds_t;
typedef __attribute__((address_space(1))) void glb_t;

// ------------------------------------------------------------------ bf16
// Each wave's work is ordered so the matrix core and the vector ALUs overlap
// inside one wave: the softmax of tile i (exp2, bf16 packing, row sums) is split
// evenly over the MFMAs of O += V P^T for tile i - 1 and those of S = K Q^T for
// tile i + 1, one score per MFMA.  There is no per-score row max: P is exp2 of
// (score - m) with a lagging running max m, and a tile whose row sum on some lane
// exceeds 256 is redone after m moves to the tile's max (rare after the first
// tile, which starts from its own max).  K / V^T tiles come through a ring of
// STAGES LDS buffers filled STAGES - 1 tiles ahead by direct loads, issued one at
// a time between the S MFMAs; loads past the last tile replay it into a buffer
// that is never read again, so the number of loads in flight is the same on
// every tile.
template <int WAVES, int STAGES>
__global__ __launch_bounds__(WAVES * 64, 1) void attn_bf16_d128(AttnParams p) {
  constexpr int K_INS = K_STAGE / 1024 / WAVES;   // 1 KB direct loads per wave per K tile
  constexpr int V_INS = V_STAGE / 1024 / WAVES;
  constexpr int LPW = K_INS + V_INS;
  constexpr int STAGE = K_STAGE + V_STAGE;
  static_assert(STAGES >= 3, "ring depth");
  extern __shared__ __attribute__((aligned(16))) char smem[];

  const int64_t nqt = (p.n_q + 32 * WAVES - 1) / (32 * WAVES);
  const int64_t total = nqt * p.B * p.heads;
  const int64_t pid = blockIdx.x;
  const int64_t full = total / 8 * 8;
  const int64_t lid = pid < full ? (pid % 8) * (full / 8) + pid / 8 : pid;
  const int64_t qt = lid % nqt, bh = lid / nqt;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ql = lane & 31, g = lane >> 5;
  const int64_t q0 = qt * 32 * WAVES + wave * 32;
  const int n_kv = static_cast<int>(p.n_kv);
  const bf16_t* Kb = p.K + bh * p.n_kv * D;
  const bf16_t* Vb = p.Vt + bh * D * p.n_kv;

  bf16x8_t qf[8];
  {
    int64_t q = q0 + ql;
    if (q >= p.n_q) q = p.n_q - 1;
    const bf16_t* qp = p.Q + (bh / p.heads) * p.q_bs + (bh % p.heads) * p.q_hs + q * p.q_rs + 8 * g;
#pragma unroll
    for (int t = 0; t < 8; ++t) qf[t] = *reinterpret_cast<const bf16x8_t*>(qp + 16 * t);
  }

  int k_row[K_INS], k_ck[K_INS], v_row[V_INS], v_ck[V_INS];
#pragma unroll
  for (int i = 0; i < K_INS; ++i) {
    k_row[i] = 4 * (i * WAVES + wave) + (lane >> 4);
    k_ck[i] = (lane & 15) ^ (k_row[i] & 15);
  }
#pragma unroll
  for (int i = 0; i < V_INS; ++i) {
    v_row[i] = 8 * (i * WAVES + wave) + (lane >> 3);
    v_ck[i] = (lane & 7) ^ ((v_row[i] >> 1) & 7);
  }
  const int ntiles = (n_kv + KT - 1) / KT;
  const int nfull = n_kv / KT;   // tiles without masked keys
  // The direct loads are written as inline assembly: the compiler's wait-count pass cannot
  // tell an LDS-DMA load's destination from the fragment reads, and with one in flight it
  // turns every LDS wait into lgkmcnt(0) (and adds a vmcnt(0) before the reads), which
  // defeats the read prefetch.  Their completion is ordered explicitly instead (vmcnt wait
  // and barrier before a tile is read; its buffer is refilled only after the next barrier).
  // (M0 is written here as in the GEMM's loads: no compiler value lives in M0 in this kernel.)
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  auto dma16 = [](const void* src, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                 :: "s"(lds_addr), "v"(src) : "memory", "m0");
  };
#pragma clang diagnostic pop
  const uint32_t smem_base = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(smem));
  // Load j (0 .. LPW - 1) of this wave's share of tile `tile`: K loads first, then V^T.
  auto issue_one = [&](int tile, int j) {
    const int kv0 = (tile < ntiles ? tile : ntiles - 1) * KT;
    const uint32_t base = smem_base + static_cast<uint32_t>((tile % STAGES) * STAGE);
    if (j < K_INS) {
      const int key = kv0 + k_row[j] < n_kv ? kv0 + k_row[j] : n_kv - 1;
      dma16(Kb + key * D + k_ck[j] * 8, __builtin_amdgcn_readfirstlane(base + (j * WAVES + wave) * 1024));
    } else {
      const int i = j - K_INS;
      const int col = kv0 + v_ck[i] * 8 < n_kv ? kv0 + v_ck[i] * 8 : n_kv - 8;
      dma16(Vb + v_row[i] * n_kv + col, __builtin_amdgcn_readfirstlane(base + K_STAGE + (i * WAVES + wave) * 1024));
    }
  };
  auto issue = [&](int tile) {
#pragma unroll
    for (int j = 0; j < LPW; ++j) issue_one(tile, j);
  };

  f32x16_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[i][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const int krow = (ql & ~12) | ((ql & 4) << 1) | ((ql & 8) >> 1);   // K row fed to MFMA row ql

  // The two halves of a tile step are written out as 16 fused steps, fenced so the
  // compiler keeps the order: each issues one MFMA, the LDS read of the fragment six
  // steps ahead, and the softmax of one score of the current tile.
  constexpr int AHEAD = 6;
  // K fragment f = (t, kb) of S^T = K Q^T: K rows 32 kb + krow, d slots 16 t + 8 g.
  auto k_frag = [&](const char* Ks, int f) {
    return *reinterpret_cast<const bf16x8_t*>(Ks + k_off(32 * (f & 1) + krow, 2 * (f >> 1) + g));
  };
  // V^T fragment f = (sl, db) of O^T += V^T P^T: V^T rows 32 db + ql, keys 16 sl + 8 g.
  auto v_frag = [&](const char* Vs, int f) {
    return *reinterpret_cast<const bf16x8_t*>(Vs + v_off(32 * (f & 3) + ql, 2 * (f >> 2) + g));
  };
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  const bf16x2_t ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
  // Score i (0..31) of a tile: s[i / 16][i % 16]; its P slot is pf[i / 8][i % 8].  The offsets
  // nm[g8] = -m (or -inf for a group of 8 keys past n_kv).  Odd scores pack the pair into its
  // P slots and add both bf16 values to the tile's row sum lt (so l sums the P that O uses).
  float e_even = 0.f;
  auto soft = [&](int i, const f32x16_t (&s)[2], bf16x8_t (&pf)[4], const float (&nm)[4], float& lt) {
    const float e = __builtin_amdgcn_exp2f(fmaf(s[i >> 4][i & 15], p.scale_log2, nm[i >> 3]));
    if (i & 1) {
      const bf16x2_t pr = {static_cast<__bf16>(e_even), static_cast<__bf16>(e)};
      pf[i >> 3][(i & 7) - 1] = pr[0];
      pf[i >> 3][i & 7] = pr[1];
      lt = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, lt, false);
    } else {
      e_even = e;
    }
  };
  auto offsets = [&](int tile, float (&nm)[4]) {
    const int kv0 = tile * KT;
#pragma unroll
    for (int gi = 0; gi < 4; ++gi) nm[gi] = kv0 + 8 * (2 * gi + g) < n_kv ? -m_run : -INFINITY;
  };
  auto mfma_o = [](f32x16_t& acc, const bf16x8_t& a, const bf16x8_t& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
  };
  // O += V P^T of tile `tile` (P in pf) with the softmax of scores 0..15 of the next tile.
  auto pv_soft = [&](int tile, const bf16x8_t (&pf)[4], const f32x16_t (&s)[2], bf16x8_t (&pn)[4],
                     const float (&nm)[4], float& lt) {
    const char* Vs = smem + (tile % STAGES) * STAGE + K_STAGE;
    bf16x8_t vf[16];
#pragma unroll
    for (int f = 0; f < AHEAD; ++f) vf[f] = v_frag(Vs, f);
#pragma unroll
    for (int f = 0; f < 16; ++f) {
      mfma_o(o[f & 3], vf[f], pf[f >> 2]);
      if (f + AHEAD < 16) vf[f + AHEAD] = v_frag(Vs, f + AHEAD);
      soft(f, s, pn, nm, lt);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  auto pv = [&](int tile, const bf16x8_t (&pf)[4]) {
    const char* Vs = smem + (tile % STAGES) * STAGE + K_STAGE;
#pragma unroll
    for (int f = 0; f < 16; ++f) mfma_o(o[f & 3], v_frag(Vs, f), pf[f >> 2]);
  };
  auto rowmax = [&](const f32x16_t (&s)[2]) {
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
    return fmaxf(mx, __shfl_xor(mx, 32, 64)) * p.scale_log2;
  };
  // S of tile `next` with the softmax of scores 16..31 of the current tile.
  auto qk_soft = [&](int next, f32x16_t (&s_nxt)[2], const f32x16_t (&s)[2], bf16x8_t (&pf)[4],
                     const float (&nm)[4], float& lt, int load_tile) {
    const char* Ks = smem + (next % STAGES) * STAGE;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s_nxt[kb][r] = 0.f;
    bf16x8_t kf[16];
#pragma unroll
    for (int f = 0; f < AHEAD; ++f) kf[f] = k_frag(Ks, f);
#pragma unroll
    for (int f = 0; f < 16; ++f) {
      s_nxt[f & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[f], qf[f >> 1], s_nxt[f & 1], 0, 0, 0);
      if (f + AHEAD < 16) kf[f + AHEAD] = k_frag(Ks, f + AHEAD);
      if (f % (16 / LPW) == 1) issue_one(load_tile, f / (16 / LPW));
      soft(16 + f, s, pf, nm, lt);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  auto qk = [&](int tile, f32x16_t (&s)[2]) {
    const char* Ks = smem + (tile % STAGES) * STAGE;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
#pragma unroll
    for (int f = 0; f < 16; ++f) s[f & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k_frag(Ks, f), qf[f >> 1], s[f & 1], 0, 0, 0);
  };
  // The running max m lags: every P of a tile is exp2 of (score - m), and a tile whose row sum
  // on some lane exceeds 256 (a score more than 8 above m, in log2 units, or enough scores near
  // it) is redone: m moves to the tile's max, O and l are rescaled, and the tile's P recomputed.
  // The first tile starts from its own max.
  auto redo = [&](int tile, const f32x16_t (&s)[2], bf16x8_t (&pf)[4], float& lt) {
    const float m_new = fmaxf(m_run, rowmax(s));
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[i][r] *= alpha;
    float nm[4];
    offsets(tile, nm);
    lt = 0.f;
#pragma unroll
    for (int i = 0; i < 32; ++i) soft(i, s, pf, nm, lt);
  };
  auto wait_next = [&]() {   // tile it + 1 has landed in every wave's view
    if constexpr (STAGES == 3) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    else asm volatile("s_waitcnt vmcnt(%0)" ::"n"((STAGES - 3) * LPW) : "memory");
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_barrier" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
  };
  // Tile it: [O += V P^T of tile it - 1 | softmax of half of tile it], wait for tile it + 1,
  // issue tile it + STAGES - 1, [S of tile it + 1 | softmax of the other half of tile it], check.
  auto iter = [&](int it, f32x16_t (&s_cur)[2], f32x16_t (&s_nxt)[2], const bf16x8_t (&p_prev)[4],
                  bf16x8_t (&p_cur)[4], bool first) {
    float nm[4];
    if (first) m_run = rowmax(s_cur);
    offsets(it, nm);
    float lt = 0.f;
    if (first) {
#pragma unroll
      for (int i = 0; i < 16; ++i) soft(i, s_cur, p_cur, nm, lt);
    } else {
      pv_soft(it - 1, p_prev, s_cur, p_cur, nm, lt);
    }
    __builtin_amdgcn_sched_barrier(0);
    wait_next();
    __builtin_amdgcn_sched_barrier(0);
    qk_soft(it + 1, s_nxt, s_cur, p_cur, nm, lt, it + STAGES - 1);   // past the last tile: replayed data, unused
    if (__any(lt > 256.0f)) redo(it, s_cur, p_cur, lt);
    l_run += lt;
  };

#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st) issue(st);
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"((STAGES - 2) * LPW) : "memory");   // tile 0 has landed
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  f32x16_t sA[2], sB[2];
  bf16x8_t pA[4], pB[4];
  qk(0, sA);
  iter(0, sA, sB, pB, pA, true);
  int it = 1;
  for (; it + 1 < ntiles; it += 2) {
    iter(it, sB, sA, pA, pB, false);
    iter(it + 1, sA, sB, pB, pA, false);
  }
  if (it < ntiles) {
    iter(it, sB, sA, pA, pB, false);
    pv(it, pB);
  } else {
    pv(ntiles - 1, pA);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // replayed loads may still target LDS

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_tot;
  // O^T blocks to row-major bf16 through LDS (the ring is free once every wave is past its last
  // tile): a lane holds 4-element pieces of one query's row, so it writes them into a per-wave
  // 32 x 132 bf16 scratch (the 264-byte stride keeps the 8-byte writes and the 16-byte reads
  // conflict-free), and each query row then leaves as 256 contiguous bytes from 16 lanes.
  constexpr int OLD = 132;
  __syncthreads();
  bf16_t* os = reinterpret_cast<bf16_t*>(smem) + wave * 32 * OLD;
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      uint2 w;
      w.x = uint32_t(f2bf(o[db][4 * u] * inv)) | (uint32_t(f2bf(o[db][4 * u + 1] * inv)) << 16);
      w.y = uint32_t(f2bf(o[db][4 * u + 2] * inv)) | (uint32_t(f2bf(o[db][4 * u + 3] * inv)) << 16);
      *reinterpret_cast<uint2*>(os + ql * OLD + 32 * db + 8 * u + 4 * g) = w;
    }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  const int64_t b = bh / p.heads, h = bh % p.heads;
  const int cl = (lane & 15) * 8;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int r = k * 4 + (lane >> 4);
    const uint4 w = *reinterpret_cast<const uint4*>(os + r * OLD + cl);
    const int64_t q = q0 + r;
    if (q >= p.n_q) continue;
    bf16_t* row;
    if (q < p.split) row = p.out0 + (b * p.split + q) * p.ldo;
    else row = p.out1 + (b * (p.n_q - p.split) + (q - p.split)) * p.ldo;
    *reinterpret_cast<uint4*>(row + h * D + cl) = w;
  }
}

// ------------------------------------------------------------------ float32
struct AttnF32Params {
  int64_t B, heads, n_q, n_kv, d;
  const float* Q; const float* K; const float* V;   // V not transposed: [B, h, n_kv, d]
  float* out0; float* out1; int64_t split; int64_t ldo;
  float scale;
  int64_t q_bs, q_hs, q_rs;
};

__global__ __launch_bounds__(64) void attn_f32_kernel(AttnF32Params p) {
  const int64_t q = static_cast<int64_t>(blockIdx.x) * 64 + threadIdx.x;
  const int64_t bh = blockIdx.y;
  if (q >= p.n_q) return;
  constexpr int MAXD = 64;
  float qv[MAXD], acc[MAXD];
  const int d = static_cast<int>(p.d);
  const float* qp = p.Q + (bh / p.heads) * p.q_bs + (bh % p.heads) * p.q_hs + q * p.q_rs;
  for (int i = 0; i < d; ++i) { qv[i] = qp[i]; acc[i] = 0.f; }
  float m = -INFINITY, l = 0.f;
  for (int64_t k = 0; k < p.n_kv; ++k) {
    const float* kp = p.K + (bh * p.n_kv + k) * d;
    float sc = 0.f;
    for (int i = 0; i < d; ++i) sc = fmaf(qv[i], kp[i], sc);
    sc *= p.scale;
    const float mn = fmaxf(m, sc);
    const float alpha = expf(m - mn), e = expf(sc - mn);
    l = l * alpha + e;
    const float* vp = p.V + (bh * p.n_kv + k) * d;
    for (int i = 0; i < d; ++i) acc[i] = fmaf(e, vp[i], acc[i] * alpha);
    m = mn;
  }
  const int64_t b = bh / p.heads, h = bh % p.heads;
  float* row = q < p.split ? p.out0 + (b * p.split + q) * p.ldo
                           : p.out1 + (b * (p.n_q - p.split) + (q - p.split)) * p.ldo;
  row += h * d;
  for (int i = 0; i < d; ++i) row[i] = acc[i] / l;
}

}  // namespace

int attention(const AttnArgs& a, hipStream_t s) {
  if (a.B == 0 || a.n_q == 0) return FF_OK;
  const bool default_q = a.q_bs == 0 && a.q_hs == 0 && a.q_rs == 0;
  const int64_t qbs = default_q ? a.heads * a.n_q * a.d : a.q_bs;
  const int64_t qhs = default_q ? a.n_q * a.d : a.q_hs;
  const int64_t qrs = default_q ? a.d : a.q_rs;
  const double flops = 4.0 * a.B * a.heads * static_cast<double>(a.n_q) * a.n_kv * a.d;
  const double esz = static_cast<double>(dtype_size(a.dtype));
  const double bytes = esz * a.B * a.heads * a.d * (2.0 * a.n_q + 2.0 * a.n_kv);
  if (a.dtype == FF_BF16) {
    if (a.d != D) return fail(FF_EUNSUPPORTED, "attention: bf16 head_dim %lld (128 required)", (long long)a.d);
    if (a.n_kv % 8 != 0) return fail(FF_EUNSUPPORTED, "attention: bf16 n_kv=%lld must be a multiple of 8", (long long)a.n_kv);
    AttnParams p{a.B, a.heads, a.n_q, a.n_kv,
                 static_cast<const bf16_t*>(a.Q), static_cast<const bf16_t*>(a.K), static_cast<const bf16_t*>(a.Vt),
                 static_cast<bf16_t*>(a.out0), static_cast<bf16_t*>(a.out1), a.split, a.ldo,
                 static_cast<float>(a.scale * 1.4426950408889634), qbs, qhs, qrs};
    constexpr int WAVES = 8, STAGES = 4, smem = STAGES * (K_STAGE + V_STAGE);
    static std::atomic<uint64_t> limit_set{0};
    FF_TRY(ensure_smem_limit(reinterpret_cast<const void*>(&attn_bf16_d128<WAVES, STAGES>), smem, limit_set));
    const int64_t tiles = (a.n_q + 32 * WAVES - 1) / (32 * WAVES) * a.B * a.heads;
    LaunchScope ls("attn_bf16_d128", s, flops, bytes);
    hipLaunchKernelGGL((attn_bf16_d128<WAVES, STAGES>), dim3(static_cast<unsigned>(tiles)), dim3(64 * WAVES), smem, s, p);
    return ls.status();
  }
  if (a.d > 64) return fail(FF_EUNSUPPORTED, "attention: f32 head_dim %lld > 64", (long long)a.d);
  if (a.B * a.heads > 65535) return fail(FF_EUNSUPPORTED, "attention: f32 needs B x heads <= 65535 (one grid row each)");
  AttnF32Params p{a.B, a.heads, a.n_q, a.n_kv, a.d,
                  static_cast<const float*>(a.Q), static_cast<const float*>(a.K), static_cast<const float*>(a.Vt),
                  static_cast<float*>(a.out0), static_cast<float*>(a.out1), a.split, a.ldo, a.scale, qbs, qhs, qrs};
  LaunchScope ls("attn_f32", s, flops, bytes);
  hipLaunchKernelGGL(attn_f32_kernel, dim3(static_cast<unsigned>((a.n_q + 63) / 64), static_cast<unsigned>(a.B * a.heads)),
                     dim3(64), 0, s, p);
  return ls.status();
}

}  // namespace ff
