// Joint (text + image) attention O = softmax(Q K^T / sqrt(d)) V, non-causal.
//
// bf16, d = 128: a flash-style kernel with online softmax in float32.  Each
// wave owns 32 queries; a workgroup of WAVES waves shares 64-key tiles of K
// and V^T staged through LDS (double-buffered, the next tile's global loads in
// flight during the current tile's math).  Both products are computed
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
#include <cstdlib>

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

// One 64-key tile: S^T = K Q^T, online softmax (masked when MASK), O^T += V^T P^T.
#define FF_ATTN_TILE(MASK)                                                                          \
  {                                                                                                 \
    const char* Ks = smem + (it % STAGES) * (K_STAGE + V_STAGE);                                     \
    const char* Vs = Ks + K_STAGE;                                                                  \
    f32x16_t s[2];                                                                                  \
    _Pragma("unroll") for (int kb = 0; kb < 2; ++kb)                                                \
      _Pragma("unroll") for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;                                \
    _Pragma("unroll") for (int t = 0; t < 8; ++t)                                                   \
      _Pragma("unroll") for (int kb = 0; kb < 2; ++kb) {                                            \
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(Ks + k_off(32 * kb + krow, 2 * t + g)); \
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[t], s[kb], 0, 0, 0);                  \
      }                                                                                             \
    if (MASK) {                                                                                     \
      /* keys come in aligned groups of 8 (n_kv % 8 == 0): one test per group */                    \
      _Pragma("unroll") for (int kb = 0; kb < 2; ++kb)                                              \
        _Pragma("unroll") for (int u = 0; u < 2; ++u) {                                             \
          const bool dead = kv0 + 32 * kb + 16 * u + 8 * g >= p.n_kv;                              \
          _Pragma("unroll") for (int j = 0; j < 8; ++j)                                             \
            if (dead) s[kb][8 * u + j] = -INFINITY;                                                 \
        }                                                                                           \
    }                                                                                               \
    float mx = -INFINITY;                                                                           \
    _Pragma("unroll") for (int kb = 0; kb < 2; ++kb)                                                \
      _Pragma("unroll") for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);                      \
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * p.scale_log2;                                          \
    if (__any(mx > m_run + 8.0f)) {                                                                 \
      const float m_new = fmaxf(m_run, mx);                                                         \
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);                                    \
      m_run = m_new;                                                                                \
      l_run *= alpha;                                                                               \
      _Pragma("unroll") for (int i = 0; i < 4; ++i)                                                 \
        _Pragma("unroll") for (int r = 0; r < 16; ++r) o[i][r] *= alpha;                            \
    }                                                                                               \
    const float neg_m = -m_run;                                                                     \
    float lsum = 0.f;                                                                               \
    bf16x8_t pf[4];                                                                                 \
    _Pragma("unroll") for (int kb = 0; kb < 2; ++kb)                                                \
      _Pragma("unroll") for (int u = 0; u < 2; ++u)                                                 \
        _Pragma("unroll") for (int j = 0; j < 8; ++j) {                                             \
          const float e = __builtin_amdgcn_exp2f(fmaf(s[kb][8 * u + j], p.scale_log2, neg_m));      \
          lsum += e;                                                                                \
          pf[2 * kb + u][j] = static_cast<__bf16>(e);                                               \
        }                                                                                           \
    l_run += lsum;                                                                                  \
    _Pragma("unroll") for (int sl = 0; sl < 4; ++sl)                                                \
      _Pragma("unroll") for (int db = 0; db < 4; ++db) {                                            \
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(Vs + v_off(32 * db + ql, 2 * sl + g)); \
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[sl], o[db], 0, 0, 0);                 \
      }                                                                                             \
  }

template <int WAVES, int STAGES>
__global__ __launch_bounds__(WAVES * 64, 8 / WAVES) void attn_bf16_d128(AttnParams p) {
  constexpr int K_INS = K_STAGE / 1024 / WAVES;   // 1 KB direct loads per wave per K tile
  constexpr int V_INS = V_STAGE / 1024 / WAVES;
  __shared__ __attribute__((aligned(16))) char smem[STAGES * (K_STAGE + V_STAGE)];

  // Workgroup -> (query tile, batch*head): ids are regrouped so the query
  // tiles of one (b, h) run on one XCD and share its L2.
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

  // Q fragments: query q0 + ql, d slots 16t + 8g .. +7.
  bf16x8_t qf[8];
  {
    int64_t q = q0 + ql;
    if (q >= p.n_q) q = p.n_q - 1;
    const bf16_t* qp = p.Q + (bh / p.heads) * p.q_bs + (bh % p.heads) * p.q_hs + q * p.q_rs + 8 * g;
#pragma unroll
    for (int t = 0; t < 8; ++t) qf[t] = *reinterpret_cast<const bf16x8_t*>(qp + 16 * t);
  }

  // Direct loads.  K: instruction i of this wave fills K rows 4(i*WAVES + wave) .. +3; lane l
  // lands at row + l/16, stored chunk l%16 = logical chunk ^ (row & 15).  V^T: instruction i
  // fills rows 8(i*WAVES + wave) .. +7; lane l lands at row + l/8, stored chunk l%8 = logical
  // chunk ^ ((row >> 1) & 7).  Keys past n_kv are clamped to valid memory and masked.
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
  auto issue = [&](int kv0, int stage) {
    char* base = smem + stage * (K_STAGE + V_STAGE);
#pragma unroll
    for (int i = 0; i < K_INS; ++i) {
      const int key = kv0 + k_row[i] < n_kv ? kv0 + k_row[i] : n_kv - 1;
      __builtin_amdgcn_global_load_lds((const glb_t*)(Kb + key * D + k_ck[i] * 8),
                                       (lds_t*)(base + (i * WAVES + wave) * 1024), 16, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < V_INS; ++i) {
      const int col = kv0 + v_ck[i] * 8 < n_kv ? kv0 + v_ck[i] * 8 : n_kv - 8;
      __builtin_amdgcn_global_load_lds((const glb_t*)(Vb + v_row[i] * n_kv + col),
                                       (lds_t*)(base + K_STAGE + (i * WAVES + wave) * 1024), 16, 0, 0);
    }
  };

  f32x16_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[i][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  // Row of K fed to MFMA row rho: bits 2 and 3 swapped.
  const int krow = (ql & ~12) | ((ql & 4) << 1) | ((ql & 8) >> 1);

  const int ntiles = (n_kv + KT - 1) / KT;
  const int nfull = n_kv / KT;   // tiles without masked keys
#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < ntiles) issue(st * KT, st);

  for (int it = 0; it < ntiles; ++it) {
    const int kv0 = it * KT;
    // tile it has landed once at most STAGES-2 younger tiles are in flight
    if (it + STAGES - 2 < ntiles) {
      if constexpr (STAGES == 3) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(K_INS + V_INS) : "memory");
      else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    } else {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    asm volatile("s_barrier" ::: "memory");
    if (it + STAGES - 1 < ntiles) issue((it + STAGES - 1) * KT, (it + STAGES - 1) % STAGES);
    if (it < nfull) FF_ATTN_TILE(false)
    else FF_ATTN_TILE(true)
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_tot;
  const int64_t q = q0 + ql;
  if (q >= p.n_q) return;
  const int64_t b = bh / p.heads, h = bh % p.heads;
  bf16_t* row;
  if (q < p.split) row = p.out0 + (b * p.split + q) * p.ldo;
  else row = p.out1 + (b * (p.n_q - p.split) + (q - p.split)) * p.ldo;
  row += h * D;
  // o[db][4u + j] is O[q, 32db + 8u + 4g + j].
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      uint2 w;
      w.x = uint32_t(f2bf(o[db][4 * u] * inv)) | (uint32_t(f2bf(o[db][4 * u + 1] * inv)) << 16);
      w.y = uint32_t(f2bf(o[db][4 * u + 2] * inv)) | (uint32_t(f2bf(o[db][4 * u + 3] * inv)) << 16);
      *reinterpret_cast<uint2*>(row + 32 * db + 8 * u + 4 * g) = w;
    }
}
#undef FF_ATTN_TILE

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
    static const char* env = getenv("FF_ATTN_WAVES");
    const int waves = (env && env[0] == '4') ? 4 : 8;
    LaunchScope ls("attn_bf16_d128", s, flops, bytes);
    static const char* envs = getenv("FF_ATTN_STAGES");
    const int stages = (envs && envs[0] == '2') ? 2 : 3;
    if (waves == 8) {
      const int64_t tiles = (a.n_q + 255) / 256 * a.B * a.heads;
      if (stages == 3) hipLaunchKernelGGL((attn_bf16_d128<8, 3>), dim3(static_cast<unsigned>(tiles)), dim3(512), 0, s, p);
      else hipLaunchKernelGGL((attn_bf16_d128<8, 2>), dim3(static_cast<unsigned>(tiles)), dim3(512), 0, s, p);
    } else {
      const int64_t tiles = (a.n_q + 127) / 128 * a.B * a.heads;
      hipLaunchKernelGGL((attn_bf16_d128<4, 2>), dim3(static_cast<unsigned>(tiles)), dim3(256), 0, s, p);
    }
    return ls.status();
  }
  if (a.d > 64) return fail(FF_EUNSUPPORTED, "attention: f32 head_dim %lld > 64", (long long)a.d);
  AttnF32Params p{a.B, a.heads, a.n_q, a.n_kv, a.d,
                  static_cast<const float*>(a.Q), static_cast<const float*>(a.K), static_cast<const float*>(a.Vt),
                  static_cast<float*>(a.out0), static_cast<float*>(a.out1), a.split, a.ldo, a.scale, qbs, qhs, qrs};
  LaunchScope ls("attn_f32", s, flops, bytes);
  hipLaunchKernelGGL(attn_f32_kernel, dim3(static_cast<unsigned>((a.n_q + 63) / 64), static_cast<unsigned>(a.B * a.heads)),
                     dim3(64), 0, s, p);
  return ls.status();
}

}  // namespace ff
