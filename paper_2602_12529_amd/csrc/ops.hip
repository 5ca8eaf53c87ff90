// Bandwidth-bound DiT pieces: adaLN modulation vectors (skinny linear),
// norm + modulate, per-head QK RMSNorm + RoPE + relayout, RoPE tables,
// prompt broadcast and the sinusoidal timestep embedding.
#include <cmath>

#include "dev.h"
#include "ff_internal.h"

namespace ff {
namespace {

// ------------------------------------------------------------------ skinny linear
// out[b, n] = act_out(sum_k W[n,k] act_in(in[b,k]) + bias[n]) (+ out[b, n] when accumulating).
// Weight-bandwidth bound.  A block of four waves owns 4 R output rows, R per wave; lanes stride
// over K in 8-element chunks.  K is walked in 512-wide slices: the block stages act_in(in[b,
// slice]) for its input rows in LDS (the activation is evaluated once per block, not once per
// wave), and each wave holds the raw weights of the next slice in flight while it multiplies the
// current one against the staged inputs.
//
// Input rows are taken kSkCap at a time, one pass per blockIdx.y.  With a row map (row_classes)
// the passes run over the classes of bitwise-equal input rows: each distinct row is computed
// once and its result written to every sample of its class, so staging and multiply-adds scale
// with the number of distinct rows.  A pass with L live rows runs the body compiled for exactly
// L (a switch on L; the kernel's registers are those of the largest body).
constexpr int kSkSlice = 512, kSkCap = 8, kSkMaxSeg = 40;
constexpr int64_t kClassMaxB = 64;   // row classes are searched for B <= 64, identity above

__device__ __forceinline__ float act_apply(int act, float x) {
  if (act == ACT_SILU) return silu_f(x);
  if (act == ACT_GELU) return gelu_tanh_f(x);
  return x;
}

// Classes of bitwise-equal rows of c [B, H] (fp32).  map (int32, 2 + 3 B entries):
//   map[0]                      U, the number of classes
//   map[1 + j], j < U           first row of class j (ascending)
//   map[1 + B + j], j <= U      start of class j in the member list
//   map[2 + 2 B + m], m < B     members, grouped by class, ascending within a class
// One block of 16 waves, one wave per row at a time.  Each row gets a 64-bit hash (a sum over
// columns of a mixed (column, bits) word, so the order of the partial sums does not matter); a
// row whose hash equals an earlier row's is compared with the first such row element by element
// and joins its class only if every bit matches (a hash collision costs a missed merge, never a
// wrong one).  For B > 64 every row is its own class (no search).
__device__ __forceinline__ uint64_t mix64(uint64_t z) {   // splitmix64 finaliser
  z += 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__global__ __launch_bounds__(1024) void row_classes_kernel(const float* __restrict__ c, int64_t B, int64_t H,
                                                           int32_t* __restrict__ map) {
  int32_t* uniq = map + 1;
  int32_t* offs = map + 1 + B;
  int32_t* memb = map + 2 + 2 * B;
  if (B > kClassMaxB) {
    for (int64_t b = threadIdx.x; b < B; b += blockDim.x) {
      uniq[b] = static_cast<int32_t>(b);
      offs[b] = static_cast<int32_t>(b);
      memb[b] = static_cast<int32_t>(b);
    }
    if (threadIdx.x == 0) { map[0] = static_cast<int32_t>(B); offs[B] = static_cast<int32_t>(B); }
    return;
  }
  __shared__ unsigned long long hs[kClassMaxB];
  __shared__ int rep[kClassMaxB], cls[kClassMaxB], cnt[kClassMaxB + 1];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6, waves = blockDim.x >> 6;
  const uint32_t* cu = reinterpret_cast<const uint32_t*>(c);
  // Lane l reads the 4-word groups l, l + 64, ... of a row (16-byte loads: H % 4 == 0 and c is
  // 16-byte aligned, checked by the host).
  for (int b = wave; b < B; b += waves) {
    unsigned long long h = 0;
#pragma unroll 12
    for (int64_t k0 = 4 * lane; k0 < H; k0 += 256) {
      const uint4 q = *reinterpret_cast<const uint4*>(cu + b * H + k0);
      const uint32_t w4[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) h += mix64(static_cast<uint64_t>(k0 + i) << 32 | w4[i]);
    }
    for (int o = 32; o > 0; o >>= 1) h += __shfl_xor(h, o, 64);
    if (lane == 0) hs[b] = h;
  }
  __syncthreads();
  if (t < B) {
    int r = t;
    for (int o = 0; o < t; ++o)
      if (hs[o] == hs[t]) { r = o; break; }
    rep[t] = r;
  }
  __syncthreads();
  for (int b = wave; b < B; b += waves) {   // confirm each candidate bit for bit
    const int r = rep[b];
    if (r == b) continue;
    bool differ = false;
#pragma unroll 12
    for (int64_t k0 = 4 * lane; k0 < H; k0 += 256) {
      const uint4 x = *reinterpret_cast<const uint4*>(cu + b * H + k0);
      const uint4 y = *reinterpret_cast<const uint4*>(cu + r * H + k0);
      differ |= x.x != y.x || x.y != y.y || x.z != y.z || x.w != y.w;
    }
    if (__ballot(differ) != 0 && lane == 0) rep[b] = b;
  }
  __syncthreads();
  if (t == 0) {
    int U = 0;
    for (int b = 0; b < B; ++b) {
      if (rep[b] == b) { uniq[U] = b; cnt[U] = 0; cls[b] = U++; }
      else cls[b] = cls[rep[b]];
      ++cnt[cls[b]];
    }
    int run = 0;
    for (int j = 0; j < U; ++j) { offs[j] = run; const int n = cnt[j]; cnt[j] = run; run += n; }
    offs[U] = run;
    for (int b = 0; b < B; ++b) memb[cnt[cls[b]]++] = b;
    map[0] = U;
  }
}

// Step ST of the halving exchange of V per-lane values (compile-time trip counts throughout, so
// the values stay in registers): lanes whose bit (32 >> ST) is set keep the upper half.
template <int V, int ST, int S>
__device__ __forceinline__ void halve_steps(float (&a)[V], int lane) {
  if constexpr (ST < S) {
    constexpr int o = 32 >> ST, half = V >> (ST + 1);
    const bool up = (lane & o) != 0;
#pragma unroll
    for (int i = 0; i < half; ++i) {
      const float send = up ? a[i] : a[i + half];
      const float keep = up ? a[i + half] : a[i];
      a[i] = keep + __shfl_xor(send, o, 64);
    }
    halve_steps<V, ST + 1, S>(a, lane);
  }
}

struct SkinnyPass {
  const float* in; int64_t ldi; int act_in;
  const void* W; const void* bias;
  float* out; int64_t ldo; int64_t N, K;
  int accumulate, act_out;
  const int32_t* rowmap; int64_t B;
};

// One pass over BC input rows: slot b is class u0 + b of the row map (or sample u0 + b); blk is
// the workgroup's index among the workgroups of this weight matrix (4 R output rows each).
template <bool BF16, int BC, int R>
__device__ __forceinline__ void skinny_pass(const SkinnyPass& a, int64_t u0, int64_t blk, float (*xs)[kSkSlice]) {
  constexpr int WORDS = BF16 ? 4 : 8;           // 32-bit words of an 8-element chunk of a weight row
  constexpr int XPT = BC * kSkSlice / 256;      // staged inputs per thread per slice (2 per row)
  static_assert(kSkSlice == 512, "two staged inputs per row and thread");
  const int64_t K = a.K, N = a.N;
  int64_t row[BC];
#pragma unroll
  for (int b = 0; b < BC; ++b) row[b] = a.rowmap ? a.rowmap[1 + u0 + b] : u0 + b;
  const int lane = threadIdx.x & 63;
  const int64_t n0 = (blk * 4 + (threadIdx.x >> 6)) * R;
  const bool active = n0 < N;   // wave-uniform
  float acc[R][BC];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int b = 0; b < BC; ++b) acc[r][b] = 0.f;
  // Everything a slice needs from memory is loaded one slice ahead: this lane's chunk of the
  // R weight rows and this thread's share of the inputs to stage.
  uint32_t raw[R][WORDS];
  float xin[XPT];
  auto fetch = [&](int64_t k0) {
    const int len = K - k0 < kSkSlice ? static_cast<int>(K - k0) : kSkSlice;
    if (len <= 0) return;
    const float* src_x = a.in + k0 + threadIdx.x;
#pragma unroll
    for (int q = 0; q < XPT; ++q) {   // row q / 2, column threadIdx.x + 256 (q % 2) of the slice
      const int j = static_cast<int>(threadIdx.x) + ((q & 1) << 8);
      xin[q] = j < len ? src_x[row[q >> 1] * a.ldi + ((q & 1) << 8)] : 0.f;
    }
    if (!active || lane * 8 >= len) return;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int64_t n = n0 + r < N ? n0 + r : N - 1;
      const uint4* src = reinterpret_cast<const uint4*>(static_cast<const char*>(a.W) + (n * K + k0 + lane * 8) * (BF16 ? 2 : 4));
#pragma unroll
      for (int h = 0; h < WORDS / 4; ++h) {
        const uint4 u = src[h];
        raw[r][4 * h] = u.x; raw[r][4 * h + 1] = u.y; raw[r][4 * h + 2] = u.z; raw[r][4 * h + 3] = u.w;
      }
    }
  };
  fetch(0);
  for (int64_t k0 = 0; k0 < K; k0 += kSkSlice) {
    const int len = K - k0 < kSkSlice ? static_cast<int>(K - k0) : kSkSlice;
    __syncthreads();   // the previous slice has been consumed
#pragma unroll
    for (int q = 0; q < XPT; ++q) xs[q >> 1][threadIdx.x + ((q & 1) << 8)] = act_apply(a.act_in, xin[q]);
    float w[R][8];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if constexpr (BF16) w[r][j] = __uint_as_float(j & 1 ? raw[r][j >> 1] & 0xffff0000u : raw[r][j >> 1] << 16);
        else w[r][j] = __uint_as_float(raw[r][j]);
      }
    fetch(k0 + kSkSlice);
    __syncthreads();
    if (active && lane * 8 < len) {
#pragma unroll
      for (int b = 0; b < BC; ++b) {
        const float4 u = *reinterpret_cast<const float4*>(&xs[b][lane * 8]);
        const float4 v = *reinterpret_cast<const float4*>(&xs[b][lane * 8 + 4]);
        const float x[8] = {u.x, u.y, u.z, u.w, v.x, v.y, v.z, v.w};
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
          for (int j = 0; j < 8; ++j) acc[r][b] = fmaf(w[r][j], x[j], acc[r][b]);
      }
    }
  }
  if (!active) return;
  // Wave-wide sums of the R x BC partial sums by halving exchanges: at each step a lane keeps the
  // half of its values that its lane bit selects and adds the partner's copy of that half, so the
  // V = R x BCP values (BCP = BC rounded up to a power of two, padded with zeros) need V - 1
  // shuffles instead of V x 6.  Afterwards lane l holds the full sum of value l >> (6 - S),
  // i.e. one (row, slot) per lane, and stores it.  Every value is summed over the same lane
  // tree (pairs differing in lane bit 32, then 16, ...), whatever its slot.
  constexpr int BCP = BC <= 1 ? 1 : BC <= 2 ? 2 : BC <= 4 ? 4 : BC <= 8 ? 8 : 16;
  constexpr int V = R * BCP;
  constexpr int S = V <= 1 ? 0 : V <= 2 ? 1 : V <= 4 ? 2 : V <= 8 ? 3 : V <= 16 ? 4 : V <= 32 ? 5 : 6;
  static_assert((1 << S) == V && S <= 6, "R x BCP must be a power of two up to 64");
  float v[V];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int b = 0; b < BCP; ++b) v[r * BCP + b] = b < BC ? acc[r][b] : 0.f;
  halve_steps<V, 0, S>(v, lane);
#pragma unroll
  for (int o = 32 >> S; o > 0; o >>= 1) v[0] += __shfl_xor(v[0], o, 64);
  const int slot = lane >> (6 - S);
  const int r = slot / BCP, b = slot % BCP;
  if (b < BC && n0 + r < N && (lane & ((1 << (6 - S)) - 1)) == 0) {
    const int64_t n = n0 + r;
    const float y = act_apply(a.act_out, v[0] + (a.bias ? ld1<BF16>(a.bias, n) : 0.f));
    int m0 = 0, m1 = 1;
    const int32_t* memb = nullptr;
    if (a.rowmap) {
      m0 = a.rowmap[1 + a.B + u0 + b];
      m1 = a.rowmap[2 + a.B + u0 + b];
      memb = a.rowmap + 2 + 2 * a.B;
    }
    for (int m = m0; m < m1; ++m) {
      float* o = a.out + (memb ? memb[m] : u0 + b) * a.ldo + n;
      *o = a.accumulate ? y + *o : y;
    }
  }
}

template <bool BF16, int R>
__device__ __forceinline__ void skinny_dispatch_live(const SkinnyPass& a, int64_t blk, float (*xs)[kSkSlice]) {
  const int64_t U = a.rowmap ? a.rowmap[0] : a.B;
  const int64_t u0 = static_cast<int64_t>(blockIdx.y) * kSkCap;
  if (u0 >= U) return;   // uniform over the block: this pass has no rows
  const int live = U - u0 < kSkCap ? static_cast<int>(U - u0) : kSkCap;
  switch (live) {
    case 1: skinny_pass<BF16, 1, R>(a, u0, blk, xs); break;
    case 2: skinny_pass<BF16, 2, R>(a, u0, blk, xs); break;
    case 3: skinny_pass<BF16, 3, R>(a, u0, blk, xs); break;
    case 4: skinny_pass<BF16, 4, R>(a, u0, blk, xs); break;
    case 5: skinny_pass<BF16, 5, R>(a, u0, blk, xs); break;
    case 6: skinny_pass<BF16, 6, R>(a, u0, blk, xs); break;
    case 7: skinny_pass<BF16, 7, R>(a, u0, blk, xs); break;
    default: skinny_pass<BF16, 8, R>(a, u0, blk, xs); break;
  }
}

template <bool BF16, int R>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void skinny_kernel(SkinnyPass a) {
  __shared__ __attribute__((aligned(16))) float xs[kSkCap][kSkSlice];
  skinny_dispatch_live<BF16, R>(a, blockIdx.x, xs);
}

// Several weight matrices against the same input rows in one launch (the modulation vectors of
// every block of a forward): workgroup x belongs to the segment s with block0[s] <= x <
// block0[s + 1].  One long weight stream instead of one short launch per matrix.
struct SkinnySegs {
  int nseg;
  int64_t block0[kSkMaxSeg + 1];
  const void* W[kSkMaxSeg];
  const void* bias[kSkMaxSeg];
  float* out[kSkMaxSeg];
  int64_t N[kSkMaxSeg];
};

template <bool BF16, int R>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void skinny_multi_kernel(SkinnyPass a,
                                                                                                  SkinnySegs g) {
  __shared__ __attribute__((aligned(16))) float xs[kSkCap][kSkSlice];
  const int64_t x = blockIdx.x;
  int sg = 0;
  while (sg + 1 < g.nseg && g.block0[sg + 1] <= x) ++sg;
  a.W = g.W[sg];
  a.bias = g.bias[sg];
  a.out = g.out[sg];
  a.N = g.N[sg];
  a.ldo = g.N[sg];
  skinny_dispatch_live<BF16, R>(a, x - g.block0[sg], xs);
}

// ------------------------------------------------------------------ norm + modulate
// One wave per row.  NCH > 0: the row is held in registers as NCH chunks of 8
// per lane (row width 512 * NCH, 16-byte aligned) and a wave walks ROWS rows,
// keeping the sample's (1 + scale) and shift for its columns in registers
// (reloaded only when the sample changes), so every global access is a
// 16-byte vector access.  NCH == 0: generic scalar path, one row per wave.
constexpr int kNormRows = 4;

template <bool BF16, int NCH>
__global__ __launch_bounds__(256) void norm_kernel(NormArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t H = a.H;
  const float invH = 1.0f / static_cast<float>(H);
  if constexpr (NCH > 0) {
    const int64_t row0 = (static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6)) * kNormRows;
    float mul[NCH][8], add[NCH][8];
    int64_t cur_b = -1;
    for (int rr = 0; rr < kNormRows; ++rr) {
      const int64_t row = row0 + rr;
      if (row >= a.rows) break;
      const int64_t b = row / a.rows_per_sample;
      if (b != cur_b) {
        cur_b = b;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          const int64_t j0 = (c * 64 + lane) * 8;
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            float4 sc = a.scale ? *reinterpret_cast<const float4*>(a.scale + b * a.mod_ld + j0 + 4 * q) : make_float4(0.f, 0.f, 0.f, 0.f);
            float4 sh = a.shift ? *reinterpret_cast<const float4*>(a.shift + b * a.mod_ld + j0 + 4 * q) : make_float4(0.f, 0.f, 0.f, 0.f);
            mul[c][4 * q] = 1.f + sc.x; mul[c][4 * q + 1] = 1.f + sc.y; mul[c][4 * q + 2] = 1.f + sc.z; mul[c][4 * q + 3] = 1.f + sc.w;
            add[c][4 * q] = sh.x; add[c][4 * q + 1] = sh.y; add[c][4 * q + 2] = sh.z; add[c][4 * q + 3] = sh.w;
          }
          if (a.w) {
            float w8[8];
            ld8<BF16>(a.w, j0, w8);
#pragma unroll
            for (int j = 0; j < 8; ++j) mul[c][j] *= w8[j];
          }
          if (a.bias) {
            float b8[8];
            ld8<BF16>(a.bias, j0, b8);
#pragma unroll
            for (int j = 0; j < 8; ++j) add[c][j] += b8[j];
          }
        }
      }
      float v[NCH][8];
#pragma unroll
      for (int c = 0; c < NCH; ++c) ld8<BF16>(a.x, row * a.ldx + (c * 64 + lane) * 8, v[c]);
      float mean = 0.f;
      if (a.norm_kind == FF_NORM_LN) {
        float sum = 0.f;
#pragma unroll
        for (int c = 0; c < NCH; ++c)
#pragma unroll
          for (int j = 0; j < 8; ++j) sum += v[c][j];
        mean = wave_sum(sum) * invH;
      }
      float ss = 0.f;
#pragma unroll
      for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float d = v[c][j] - mean;
          ss = fmaf(d, d, ss);
        }
      const float rstd = rsqrtf(wave_sum(ss) * invH + a.eps);
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        float o[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] = fmaf((v[c][j] - mean) * rstd, mul[c][j], add[c][j]);
        st8<BF16>(a.y, row * a.ldy + (c * 64 + lane) * 8, o);
      }
    }
  } else {
    const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
    if (row >= a.rows) return;
    const int64_t b = row / a.rows_per_sample;
    const float* sh = a.shift ? a.shift + b * a.mod_ld : nullptr;
    const float* sc = a.scale ? a.scale + b * a.mod_ld : nullptr;
    auto finish = [&](int64_t j, float xn) {
      float mul = sc ? 1.0f + sc[j] : 1.0f;
      if (a.w) mul *= ld1<BF16>(a.w, j);
      float add = sh ? sh[j] : 0.0f;
      if (a.bias) add += ld1<BF16>(a.bias, j);
      return fmaf(xn, mul, add);
    };
    float mean = 0.f;
    if (a.norm_kind == FF_NORM_LN) {
      float sum = 0.f;
      for (int64_t j = lane; j < H; j += 64) sum += ld1<BF16>(a.x, row * a.ldx + j);
      mean = wave_sum(sum) * invH;
    }
    float ss = 0.f;
    for (int64_t j = lane; j < H; j += 64) {
      const float d = ld1<BF16>(a.x, row * a.ldx + j) - mean;
      ss = fmaf(d, d, ss);
    }
    const float rstd = rsqrtf(wave_sum(ss) * invH + a.eps);
    for (int64_t j = lane; j < H; j += 64)
      st1<BF16>(a.y, row * a.ldy + j, finish(j, (ld1<BF16>(a.x, row * a.ldx + j) - mean) * rstd));
  }
}

// bf16 fast path: a block of 4 waves normalises 4 RPW rows of one sample (32, or 8 when
// there are too few rows to give every CU a block).  The sample's (1 + scale) and shift are
// staged once in LDS; each wave walks RPW rows with the next row's loads issued before the
// current row is finished.  Rows are read with non-temporal loads (each is read once here and
// not again until its cached copy would long be gone): 11% faster on 32768 x 3072 rows read from
// HBM, within noise in the rollout, where the previous GEMM has just written them; non-temporal
// stores as well were slower.
template <int NCH, int RPW>
__global__ __launch_bounds__(256) void norm_lds_kernel(NormArgs a) {
  extern __shared__ __attribute__((aligned(16))) float mod_s[];   // [2][H]: mul, add
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t H = a.H;
  const int64_t r0 = static_cast<int64_t>(blockIdx.x) * 4 * RPW;
  const int64_t b = r0 / a.rows_per_sample;
  float* mul_s = mod_s;
  float* add_s = mod_s + H;
  const float invH = 1.0f / static_cast<float>(H);
  const bf16_t* __restrict__ xp = static_cast<const bf16_t*>(a.x);
  bf16_t* __restrict__ yp = static_cast<bf16_t*>(a.y);
  const int64_t rw = r0 + wave * RPW;
  float v[NCH][8], nx[NCH][8];
  if (rw < a.rows) {   // the first row is in flight while the modulation vectors are staged
#pragma unroll
    for (int c = 0; c < NCH; ++c) ld8_nt<true>(xp, rw * a.ldx + (c * 64 + lane) * 8, v[c]);
  }
  for (int64_t j = threadIdx.x * 4; j < H; j += 1024) {
    float4 sc = a.scale ? *reinterpret_cast<const float4*>(a.scale + b * a.mod_ld + j) : make_float4(0.f, 0.f, 0.f, 0.f);
    float4 sh = a.shift ? *reinterpret_cast<const float4*>(a.shift + b * a.mod_ld + j) : make_float4(0.f, 0.f, 0.f, 0.f);
    *reinterpret_cast<float4*>(mul_s + j) = make_float4(1.f + sc.x, 1.f + sc.y, 1.f + sc.z, 1.f + sc.w);
    *reinterpret_cast<float4*>(add_s + j) = sh;
  }
  __syncthreads();
  for (int rr = 0; rr < RPW; ++rr) {
    const int64_t row = rw + rr;
    if (row >= a.rows) break;
    const bool more = rr + 1 < RPW && row + 1 < a.rows;
    if (more) {
#pragma unroll
      for (int c = 0; c < NCH; ++c) ld8_nt<true>(xp, (row + 1) * a.ldx + (c * 64 + lane) * 8, nx[c]);
    }
    float mean = 0.f;
    if (a.norm_kind == FF_NORM_LN) {
      float sum = 0.f;
#pragma unroll
      for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int j = 0; j < 8; ++j) sum += v[c][j];
      mean = wave_sum(sum) * invH;
    }
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float d = v[c][j] - mean;
        ss = fmaf(d, d, ss);
      }
    const float rstd = rsqrtf(wave_sum(ss) * invH + a.eps);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int j0 = (c * 64 + lane) * 8;
      const float4 m0 = *reinterpret_cast<const float4*>(mul_s + j0), m1 = *reinterpret_cast<const float4*>(mul_s + j0 + 4);
      const float4 a0 = *reinterpret_cast<const float4*>(add_s + j0), a1 = *reinterpret_cast<const float4*>(add_s + j0 + 4);
      const float mu[8] = {m0.x, m0.y, m0.z, m0.w, m1.x, m1.y, m1.z, m1.w};
      const float ad[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
      float o[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] = fmaf((v[c][j] - mean) * rstd, mu[j], ad[j]);
      st8<true>(yp, row * a.ldy + j0, o);
    }
    if (more) {
#pragma unroll
      for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int j = 0; j < 8; ++j) v[c][j] = nx[c][j];
    }
  }
}

template <bool BF16>
int norm_dispatch(const NormArgs& a, hipStream_t s) {
  int nch = 0;
  const bool mod_ok = (!a.shift || (aligned16(a.shift) && a.mod_ld % 4 == 0)) &&
                      (!a.scale || (aligned16(a.scale) && a.mod_ld % 4 == 0)) &&
                      (!a.w || aligned16(a.w)) && (!a.bias || aligned16(a.bias));
  const bool fits = a.H % 512 == 0 && a.ldx % 8 == 0 && a.ldy % 8 == 0 && aligned16(a.x) && aligned16(a.y) && mod_ok;
  if (BF16 && fits) nch = static_cast<int>(a.H / 512);
  if (nch > 8) nch = 0;
  const int64_t block_rows = a.rows >= 64 * 512 ? 64 : a.rows >= 32 * 512 ? 32 : 8;
  const bool one_sample_blocks = a.rows_per_sample % block_rows == 0 || a.rows <= a.rows_per_sample;
  if (BF16 && nch > 0 && nch <= 6 && one_sample_blocks && !a.w && !a.bias) {
    const dim3 grid(static_cast<unsigned>((a.rows + block_rows - 1) / block_rows));
    const size_t shm = 2 * a.H * sizeof(float);
    switch (nch * 100 + static_cast<int>(block_rows)) {
#define FF_NL(N, R) case N * 100 + R: hipLaunchKernelGGL((norm_lds_kernel<N, R / 4>), grid, dim3(256), shm, s, a); return FF_OK;
      FF_NL(1, 32) FF_NL(2, 32) FF_NL(3, 32) FF_NL(4, 32) FF_NL(5, 32) FF_NL(6, 32)
      FF_NL(1, 8) FF_NL(2, 8) FF_NL(3, 8) FF_NL(4, 8) FF_NL(5, 8) FF_NL(6, 8)
      FF_NL(1, 64) FF_NL(2, 64) FF_NL(3, 64) FF_NL(4, 64) FF_NL(5, 64) FF_NL(6, 64)
#undef FF_NL
    }
  }
  const dim3 grid_rows(static_cast<unsigned>((a.rows + 4 * kNormRows - 1) / (4 * kNormRows)));
  switch (nch) {
#define FF_NM(N) case N: hipLaunchKernelGGL((norm_kernel<BF16, N>), grid_rows, dim3(256), 0, s, a); break;
    FF_NM(1) FF_NM(2) FF_NM(3) FF_NM(4) FF_NM(5) FF_NM(6) FF_NM(7) FF_NM(8)
#undef FF_NM
    default:
      hipLaunchKernelGGL((norm_kernel<BF16, 0>), dim3(static_cast<unsigned>((a.rows + 3) / 4)), dim3(256), 0, s, a);
      break;
  }
  return FF_OK;
}

// ------------------------------------------------------------------ QK norm + RoPE + relayout
// A block handles 64 tokens of one head of one sample; each wave walks 16
// tokens, lane p owning the rotation pair (2p, 2p+1).  Q and K go to
// [B, h, n_joint, d]; V goes transposed to [B, h, d, n_joint] through LDS so
// its rows are written 128 bytes at a time.
constexpr int kRopeTok = 64;

template <bool BF16>
__global__ __launch_bounds__(256) void qk_rope_kernel(QkvArgs a) {
  __shared__ float vs[kRopeTok][130];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kRopeTok;
  const int h = blockIdx.y;
  const int64_t b = blockIdx.z;
  const int d = a.d, half = d / 2;
  const bool active = lane < half;
  const float inv_d = 1.0f / static_cast<float>(d);
  for (int tt = wave; tt < kRopeTok; tt += 4) {
    const int64_t i = t0 + tt;
    if (i >= a.n_tok) break;
    const int64_t src = (b * a.src_rows + i) * a.ld + static_cast<int64_t>(h) * d + 2 * lane;
    const int64_t jn = a.tok_offset + i;
    const int64_t dst = ((b * a.heads + h) * a.n_joint + jn) * d + 2 * lane;
    float2 cs = make_float2(1.f, 0.f);
    if (a.rope && active) cs = a.rope[i * half + lane];
#pragma unroll
    for (int which = 0; which < 2; ++which) {
      const void* srcp = which == 0 ? a.q : a.k;
      const void* wn = which == 0 ? a.q_w : a.k_w;
      void* dstp = which == 0 ? a.Q : a.Kd;
      float x0 = 0.f, x1 = 0.f;
      if (active) { x0 = ld1<BF16>(srcp, src); x1 = ld1<BF16>(srcp, src + 1); }
      if (a.apply_norm) {
        const float rstd = rsqrtf(wave_sum(x0 * x0 + x1 * x1) * inv_d + a.eps);
        if (active) {
          x0 = x0 * rstd * ld1<BF16>(wn, 2 * lane);
          x1 = x1 * rstd * ld1<BF16>(wn, 2 * lane + 1);
        }
      }
      if (active) {
        const float y0 = x0 * cs.x - x1 * cs.y;
        const float y1 = x0 * cs.y + x1 * cs.x;
        st1<BF16>(dstp, dst, y0);
        st1<BF16>(dstp, dst + 1, y1);
      }
    }
    if (active) {
      float v0 = ld1<BF16>(a.v, src), v1 = ld1<BF16>(a.v, src + 1);
      if (a.v_transposed) {
        vs[tt][2 * lane] = v0;
        vs[tt][2 * lane + 1] = v1;
      } else {
        st1<BF16>(a.Vt, dst, v0);
        st1<BF16>(a.Vt, dst + 1, v1);
      }
    }
  }
  if (!a.v_transposed) return;
  __syncthreads();
  // Vt[b, h, dd, tok_offset + t0 + tt]
  const int64_t ntok = (a.n_tok - t0) < kRopeTok ? (a.n_tok - t0) : kRopeTok;
  const int64_t col0 = a.tok_offset + t0;
  for (int e = threadIdx.x; e < d * kRopeTok; e += 256) {
    const int dd = e / kRopeTok, tt = e % kRopeTok;
    if (tt < ntok) {
      const int64_t o = ((b * a.heads + h) * d + dd) * a.n_joint + col0 + tt;
      st1<BF16>(a.Vt, o, vs[tt][dd]);
    }
  }
}

// bf16, d = 128 fast path: 16 lanes per token, 8 consecutive elements per lane,
// so every load/store is 16 bytes; the per-head RMS reduction runs over the 16
// lanes of a token.  A block covers 64 tokens of one head; V^T leaves through
// an LDS transpose as 16-byte row segments.
__global__ __launch_bounds__(256) void qk_rope_vec_kernel(QkvArgs a) {
  __shared__ bf16_t vt[128][72];
  const int t = threadIdx.x, c = t & 15, tr = t >> 4;
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kRopeTok;
  const int h = blockIdx.y;
  const int64_t b = blockIdx.z;
  float qw[8], kw[8];
  if (a.apply_norm) {
    // per-head weights [128], or full-width weights [H] (this head's slice) with precomputed sums
    const int64_t wo = (a.sumsq ? static_cast<int64_t>(h) * 128 : 0) + c * 8;
    ld8<true>(a.q_w, wo, qw);
    ld8<true>(a.k_w, wo, kw);
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) qw[j] = kw[j] = 1.0f;
  }
  const int64_t out_head = (b * a.heads + h) * a.n_joint;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int tt = tr + 16 * i;
    const int64_t tok_raw = t0 + tt;
    const bool live = tok_raw < a.n_tok;
    const int64_t tok = live ? tok_raw : a.n_tok - 1;
    const int64_t src = (b * a.src_rows + tok) * a.ld + static_cast<int64_t>(h) * 128 + c * 8;
    float cs[8];   // (cos, sin) of pairs 4c .. 4c+3
    if (a.rope) {
      const float4* rp = reinterpret_cast<const float4*>(a.rope + tok * 64 + c * 4);
      const float4 r0 = rp[0], r1 = rp[1];
      cs[0] = r0.x; cs[1] = r0.y; cs[2] = r0.z; cs[3] = r0.w; cs[4] = r1.x; cs[5] = r1.y; cs[6] = r1.z; cs[7] = r1.w;
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) { cs[2 * j] = 1.f; cs[2 * j + 1] = 0.f; }
    }
    const int64_t dst = (out_head + a.tok_offset + tok) * 128 + c * 8;
    // Full-width norm: the row's sums of q^2 and k^2 over all H, from the projection's partial sums
    // (added in a fixed order, the same in every head's block).
    // Each of the token's 16 threads adds every 16th partial sum, then four exchanges (the same
    // fixed order in every block) give all 16 the totals.
    float fw_ss[2] = {0.f, 0.f};
    if (a.sumsq) {
      const float* ps = a.sumsq + (b * a.src_rows + tok) * a.sumsq_parts;
      const int64_t half = a.sumsq_parts / 2;
      for (int64_t j = c; j < half; j += 16) {
        fw_ss[0] += ps[j];
        fw_ss[1] += ps[half + j];
      }
#pragma unroll
      for (int w = 0; w < 2; ++w) {
        fw_ss[w] += __shfl_xor(fw_ss[w], 8, 64);
        fw_ss[w] += __shfl_xor(fw_ss[w], 4, 64);
        fw_ss[w] += __shfl_xor(fw_ss[w], 2, 64);
        fw_ss[w] += __shfl_xor(fw_ss[w], 1, 64);
      }
    }
#pragma unroll
    for (int which = 0; which < 2; ++which) {
      float x[8];
      ld8<true>(which == 0 ? a.q : a.k, src, x);
      float rstd = 1.0f;
      if (a.sumsq) {
        rstd = rsqrtf(fw_ss[which] / static_cast<float>(a.heads * 128) + a.eps);
      } else {
        float ss = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) ss = fmaf(x[j], x[j], ss);
        ss += __shfl_xor(ss, 8, 64);
        ss += __shfl_xor(ss, 4, 64);
        ss += __shfl_xor(ss, 2, 64);
        ss += __shfl_xor(ss, 1, 64);
        if (a.apply_norm) rstd = rsqrtf(ss * (1.0f / 128.0f) + a.eps);
      }
      const float* w = which == 0 ? qw : kw;
      float y[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float x0 = x[2 * j] * rstd * w[2 * j], x1 = x[2 * j + 1] * rstd * w[2 * j + 1];
        y[2 * j] = x0 * cs[2 * j] - x1 * cs[2 * j + 1];
        y[2 * j + 1] = x0 * cs[2 * j + 1] + x1 * cs[2 * j];
      }
      if (live) st8<true>(which == 0 ? a.Q : a.Kd, dst, y);
    }
    const uint4 vv = *reinterpret_cast<const uint4*>(static_cast<const bf16_t*>(a.v) + src);
    const uint32_t w4[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      vt[c * 8 + 2 * j][tt] = bf16_t(w4[j] & 0xffffu);
      vt[c * 8 + 2 * j + 1][tt] = bf16_t(w4[j] >> 16);
    }
  }
  __syncthreads();
  // V^T rows: thread -> (d row t/2, 32 tokens starting at 32 (t&1)), 16-byte stores.
  const int dd = t >> 1, th = (t & 1) * 32;
  bf16_t* vrow = static_cast<bf16_t*>(a.Vt) + ((b * a.heads + h) * 128 + dd) * a.n_joint + a.tok_offset + t0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int tt = th + 8 * q;
    if (t0 + tt < a.n_tok) *reinterpret_cast<uint4*>(vrow + tt) = *reinterpret_cast<const uint4*>(&vt[dd][tt]);
  }
}

__global__ void rope_table_kernel(float2* out, int64_t N, int rows, int cols, int half, int b0, int b1,
                                  int w0, int w1, int w2, double theta) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= N * half) return;
  const int64_t n = e / half;
  const int p = static_cast<int>(e % half);
  const int64_t pos[3] = {n / (static_cast<int64_t>(rows) * cols), (n / cols) % rows, n % cols};
  int axis, i, width;
  if (p < b0) { axis = 0; i = p; width = w0; }
  else if (p < b1) { axis = 1; i = p - b0; width = w1; }
  else { axis = 2; i = p - b1; width = w2; }
  const double ang = static_cast<double>(pos[axis]) * pow(theta, -2.0 * i / width);
  out[e] = make_float2(static_cast<float>(cos(ang)), static_cast<float>(sin(ang)));
}

template <bool BF16>
__global__ void gather_kernel(const void* __restrict__ in, const int32_t* __restrict__ idx, int64_t n_src,
                              void* __restrict__ out, int64_t per, int64_t total) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= total) return;
  const int64_t b = e / per, r = e % per;
  const int64_t src = idx ? idx[b] : b;
  const float v = (src >= 0 && src < n_src) ? ld1<BF16>(in, src * per + r) : 0.f;
  st1<BF16>(out, e, v);
}

__global__ void temb_kernel(const float* __restrict__ t, float* __restrict__ out, int64_t B) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= B * 128) return;
  const int64_t b = e / 128;
  const int j = static_cast<int>(e % 128);
  const double arg = 1000.0 * static_cast<double>(t[b]) * pow(10000.0, -static_cast<double>(j) / 128.0);
  out[b * 256 + j] = static_cast<float>(cos(arg));
  out[b * 256 + 128 + j] = static_cast<float>(sin(arg));
}

template <bool BF16>
__global__ void to_f32_kernel(const void* __restrict__ in, float* __restrict__ out, int64_t n) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e < n) out[e] = ld1<BF16>(in, e);
}

// out[b, r, j] = table[r, j] + e[b, r, j]  (WAN modulation: E_block + e(t))
template <bool BF16>
__global__ void add_table_kernel(const void* __restrict__ table, const float* __restrict__ e,
                                 float* __restrict__ out, int64_t B, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= B * n) return;
  out[i] = ld1<BF16>(table, i % n) + e[i];
}

unsigned blocks_for(int64_t n, int t = 256) { return static_cast<unsigned>((n + t - 1) / t); }


// Row quantisation to OCP E4M3, one workgroup per row: the row's absolute maximum (exact in
// float32), then codes = RNE(x * fl32(448 / amax)) by the hardware conversion (round to nearest
// even, the sign kept on values that round to zero) and d = fl32(amax / 448).  Eight elements
// per thread and step: 16 (bf16) or 32 (f32) bytes in, 8 bytes out.
template <bool BF16>
__global__ __launch_bounds__(256) void quantize_fp8_kernel(const void* x, int64_t ldx, uint8_t* q, int64_t ldq, float* d,
                                                           int64_t cols) {
  __shared__ float part[4];
  const int64_t r = blockIdx.x;
  const int tid = threadIdx.x;
  const int64_t n8 = cols / 8;
  float amax = 0.f;   // a NaN counts as +inf, so that any non-finite entry marks the row
  for (int64_t c = tid; c < n8; c += 256) {
    float v[8];
    ld8<BF16>(x, r * ldx + c * 8, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) amax = fmaxf(amax, __builtin_isnan(v[e]) ? INFINITY : fabsf(v[e]));
  }
  amax = wave_max(amax);
  if ((tid & 63) == 0) part[tid >> 6] = amax;
  __syncthreads();
  amax = fmaxf(fmaxf(part[0], part[1]), fmaxf(part[2], part[3]));
  // Rows below 448 * 2^-126 (zero rows included) are zero rows: codes 0, d = 0.  A row with an
  // infinity or a NaN: NaN code 0x7f everywhere, d = NaN.
  constexpr float kAmin = 448.0f * 0x1p-126f;
  const bool tiny = amax < kAmin, nonfinite = amax == INFINITY;
  if (tid == 0) d[r] = nonfinite ? __uint_as_float(0x7fc00000u) : tiny ? 0.f : amax / 448.0f;
  uint8_t* qr = q + r * ldq;
  if (tiny || nonfinite) {
    const uint32_t fill = nonfinite ? 0x7f7f7f7fu : 0u;
    for (int64_t c = tid; c < n8; c += 256) *reinterpret_cast<uint2*>(qr + c * 8) = make_uint2(fill, fill);
    return;
  }
  const float mult = 448.0f / amax;
  for (int64_t c = tid; c < n8; c += 256) {
    float v[8];
    ld8<BF16>(x, r * ldx + c * 8, v);
    int w0 = __builtin_amdgcn_cvt_pk_fp8_f32(v[0] * mult, v[1] * mult, 0, false);
    w0 = __builtin_amdgcn_cvt_pk_fp8_f32(v[2] * mult, v[3] * mult, w0, true);
    int w1 = __builtin_amdgcn_cvt_pk_fp8_f32(v[4] * mult, v[5] * mult, 0, false);
    w1 = __builtin_amdgcn_cvt_pk_fp8_f32(v[6] * mult, v[7] * mult, w1, true);
    *reinterpret_cast<uint2*>(qr + c * 8) = make_uint2(static_cast<uint32_t>(w0), static_cast<uint32_t>(w1));
  }
}

}  // namespace

int64_t row_classes_ints(int64_t B) { return 2 + 3 * B; }

int row_classes(const float* c, int64_t B, int64_t H, int32_t* map, hipStream_t s) {
  if (B == 0) return FF_OK;
  if (H % 4 || !aligned16(c)) return fail(FF_EUNSUPPORTED, "row_classes: H=%lld must be a multiple of 4, c 16-byte aligned", (long long)H);
  LaunchScope ls("row_classes", s, 0.0, 4.0 * (B * H + row_classes_ints(B)));
  hipLaunchKernelGGL(row_classes_kernel, dim3(1), dim3(1024), 0, s, c, B, H, map);
  return ls.status();
}

int skinny_linear(const SkinnyArgs& a, hipStream_t s) {
  if (a.B == 0 || a.N == 0) return FF_OK;
  if (a.K % 8 != 0 || a.ldi % 4 != 0) return fail(FF_EUNSUPPORTED, "skinny_linear: K=%lld must be a multiple of 8", (long long)a.K);
  LaunchScope ls("skinny_linear", s, 2.0 * a.B * a.N * a.K,
                 static_cast<double>(dtype_size(a.dtype)) * a.N * a.K + 4.0 * a.B * (a.K + a.N));
  // R output rows per wave: 4 for bf16 weights, 2 for fp32 (twice the words per chunk).
  const SkinnyPass k{a.in, a.ldi, a.act_in, a.W, a.bias, a.out, a.ldo, a.N, a.K, a.accumulate, a.act_out, a.rowmap, a.B};
  const int R = a.dtype == FF_BF16 ? 4 : 2;
  const dim3 grid(static_cast<unsigned>((a.N + 4 * R - 1) / (4 * R)), static_cast<unsigned>((a.B + kSkCap - 1) / kSkCap));
  if (a.dtype == FF_BF16) hipLaunchKernelGGL((skinny_kernel<true, 4>), grid, dim3(256), 0, s, k);
  else hipLaunchKernelGGL((skinny_kernel<false, 2>), grid, dim3(256), 0, s, k);
  return ls.status();
}

int skinny_linear_multi(const SkinnyArgs& a, const SkinnySeg* segs, int nseg, hipStream_t s) {
  if (a.B == 0 || nseg == 0) return FF_OK;
  if (a.K % 8 != 0 || a.ldi % 4 != 0) return fail(FF_EUNSUPPORTED, "skinny_linear: K=%lld must be a multiple of 8", (long long)a.K);
  double flops = 0.0, bytes = 0.0;
  for (int i = 0; i < nseg; ++i) {
    flops += 2.0 * a.B * segs[i].N * a.K;
    bytes += static_cast<double>(dtype_size(a.dtype)) * segs[i].N * a.K + 4.0 * a.B * (a.K + segs[i].N);
  }
  LaunchScope ls("skinny_linear", s, flops, bytes);
  const int R = a.dtype == FF_BF16 ? 4 : 2;
  const SkinnyPass k{a.in, a.ldi, a.act_in, nullptr, nullptr, nullptr, 0, 0, a.K, a.accumulate, a.act_out, a.rowmap, a.B};
  for (int first = 0; first < nseg; first += kSkMaxSeg) {
    SkinnySegs g{};
    g.nseg = nseg - first < kSkMaxSeg ? nseg - first : kSkMaxSeg;
    int64_t blocks = 0;
    for (int i = 0; i < g.nseg; ++i) {
      const SkinnySeg& sg = segs[first + i];
      g.block0[i] = blocks;
      g.W[i] = sg.W; g.bias[i] = sg.bias; g.out[i] = sg.out; g.N[i] = sg.N;
      blocks += (sg.N + 4 * R - 1) / (4 * R);
    }
    g.block0[g.nseg] = blocks;
    if (blocks == 0) continue;
    const dim3 grid(static_cast<unsigned>(blocks), static_cast<unsigned>((a.B + kSkCap - 1) / kSkCap));
    if (a.dtype == FF_BF16) hipLaunchKernelGGL((skinny_multi_kernel<true, 4>), grid, dim3(256), 0, s, k, g);
    else hipLaunchKernelGGL((skinny_multi_kernel<false, 2>), grid, dim3(256), 0, s, k, g);
  }
  return ls.status();
}

int quantize_fp8(int dtype, const void* x, int64_t ldx, void* q, int64_t ldq, float* d, int64_t rows, int64_t cols,
                 hipStream_t s) {
  if (rows == 0) return FF_OK;
  LaunchScope ls("quantize_fp8", s, 0.0, (dtype_size(dtype) + 1.0) * rows * cols + 4.0 * rows);
  if (dtype == FF_BF16)
    hipLaunchKernelGGL(quantize_fp8_kernel<true>, dim3(static_cast<unsigned>(rows)), dim3(256), 0, s, x, ldx,
                       static_cast<uint8_t*>(q), ldq, d, cols);
  else
    hipLaunchKernelGGL(quantize_fp8_kernel<false>, dim3(static_cast<unsigned>(rows)), dim3(256), 0, s, x, ldx,
                       static_cast<uint8_t*>(q), ldq, d, cols);
  return ls.status();
}

int norm_modulate(const NormArgs& a, hipStream_t s) {
  if (a.rows == 0) return FF_OK;
  LaunchScope ls("norm_modulate", s, 0.0, 2.0 * dtype_size(a.dtype) * a.rows * a.H);
  FF_TRY(a.dtype == FF_BF16 ? norm_dispatch<true>(a, s) : norm_dispatch<false>(a, s));
  return ls.status();
}

int qk_norm_rope(const QkvArgs& a, hipStream_t s) {
  if (a.B == 0 || a.n_tok == 0) return FF_OK;
  if (a.rope && a.rope_from > 0) {   // unrotated leading tokens, then the rotated rest: two passes
    const int64_t lead = a.rope_from < a.n_tok ? a.rope_from : a.n_tok;
    const size_t off = static_cast<size_t>(lead) * a.ld * dtype_size(a.dtype);
    QkvArgs head = a, tail = a;
    head.n_tok = lead; head.rope = nullptr; head.rope_from = 0;
    tail.n_tok = a.n_tok - lead; tail.tok_offset = a.tok_offset + lead; tail.rope_from = 0;
    tail.q = static_cast<const char*>(a.q) + off;
    tail.k = static_cast<const char*>(a.k) + off;
    tail.v = static_cast<const char*>(a.v) + off;
    FF_TRY(qk_norm_rope(head, s));
    return qk_norm_rope(tail, s);
  }
  if (a.d > 128 || a.d % 2) return fail(FF_EUNSUPPORTED, "qk_norm_rope: head_dim %d", a.d);
  dim3 grid(blocks_for(a.n_tok, kRopeTok), static_cast<unsigned>(a.heads), static_cast<unsigned>(a.B));
  const bool vec = a.dtype == FF_BF16 && a.d == 128 && a.v_transposed && (!a.full_width_norm || a.sumsq) &&
                   a.ld % 8 == 0 && aligned16(a.q) && aligned16(a.k) && aligned16(a.v) && aligned16(a.Q) &&
                   aligned16(a.Kd) && aligned16(a.Vt) && (!a.apply_norm || (aligned16(a.q_w) && aligned16(a.k_w))) &&
                   (!a.rope || aligned16(a.rope)) && a.n_joint % 8 == 0 && a.tok_offset % 8 == 0 && a.n_tok % 8 == 0;
  if (a.sumsq && !(vec && a.full_width_norm && a.apply_norm && a.sumsq_parts > 0 && a.sumsq_parts % 2 == 0))
    return fail(FF_EUNSUPPORTED, "qk_norm_rope: precomputed sums need the vector path and the full-width norm");
  LaunchScope ls("qk_norm_rope", s, 0.0, 6.0 * dtype_size(a.dtype) * a.B * a.n_tok * a.heads * a.d);
  if (vec) hipLaunchKernelGGL(qk_rope_vec_kernel, grid, dim3(256), 0, s, a);
  else if (a.dtype == FF_BF16) hipLaunchKernelGGL(qk_rope_kernel<true>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(qk_rope_kernel<false>, grid, dim3(256), 0, s, a);
  return ls.status();
}

int rope_table(float2* out, const int32_t grid[3], int d, const int32_t axes[3], double theta, hipStream_t s) {
  const int64_t N = static_cast<int64_t>(grid[0]) * grid[1] * grid[2];
  const int half = d / 2;
  LaunchScope ls("rope_table", s, 0.0, 8.0 * N * half);
  hipLaunchKernelGGL(rope_table_kernel, dim3(blocks_for(N * half)), dim3(256), 0, s, out, N, grid[1], grid[2],
                     half, axes[0] / 2, (axes[0] + axes[1]) / 2, axes[0], axes[1], axes[2], theta);
  return ls.status();
}

int gather_rows(int dtype, const void* in, const int32_t* idx, int64_t n_src, void* out, int64_t B,
                int64_t rows_per, int64_t width, hipStream_t s) {
  const int64_t per = rows_per * width, total = B * per;
  if (total == 0) return FF_OK;
  LaunchScope ls("gather_rows", s, 0.0, 2.0 * dtype_size(dtype) * total);
  if (dtype == FF_BF16) hipLaunchKernelGGL(gather_kernel<true>, dim3(blocks_for(total)), dim3(256), 0, s, in, idx, n_src, out, per, total);
  else hipLaunchKernelGGL(gather_kernel<false>, dim3(blocks_for(total)), dim3(256), 0, s, in, idx, n_src, out, per, total);
  return ls.status();
}

int timestep_sinusoid(const float* t, float* out, int64_t B, hipStream_t s) {
  LaunchScope ls("timestep_sinusoid", s, 0.0, 4.0 * B * 257);
  hipLaunchKernelGGL(temb_kernel, dim3(blocks_for(B * 128)), dim3(256), 0, s, t, out, B);
  return ls.status();
}

int cast_to_f32(int dtype, const void* in, float* out, int64_t n, hipStream_t s) {
  if (n == 0) return FF_OK;
  LaunchScope ls("to_f32", s, 0.0, (dtype_size(dtype) + 4.0) * n);
  if (dtype == FF_BF16) hipLaunchKernelGGL(to_f32_kernel<true>, dim3(blocks_for(n)), dim3(256), 0, s, in, out, n);
  else hipLaunchKernelGGL(to_f32_kernel<false>, dim3(blocks_for(n)), dim3(256), 0, s, in, out, n);
  return ls.status();
}

// Streaming probes (measurement only): read-only, write-only or copy of n 16-byte chunks, four
// chunks in flight per thread in a grid-stride loop; NT selects non-temporal accesses.  The
// read-only probe folds what it reads into one 16-byte word per workgroup (out[blockIdx.x]) so
// the loads are kept.
typedef unsigned int sp_u32x4 __attribute__((ext_vector_type(4)));
template <int MODE, bool NT>
__global__ __launch_bounds__(256) void stream_kernel(const sp_u32x4* __restrict__ src, sp_u32x4* __restrict__ dst,
                                                     int64_t n) {
  constexpr int U = 4;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * 256 * U;
  sp_u32x4 acc = {0u, 0u, 0u, 0u};
  const sp_u32x4 pattern = {0x3f800000u, 0u, 0x3f800000u, 0u};
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 * U + threadIdx.x; i < n; i += stride) {
    sp_u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t j = i + u * 256;
      if (MODE != 1 && j < n) v[u] = NT ? __builtin_nontemporal_load(src + j) : src[j];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t j = i + u * 256;
      if (j >= n) continue;
      if (MODE == 0) {
        acc ^= v[u];
      } else {
        const sp_u32x4 w = MODE == 1 ? pattern : v[u];
        if (NT) __builtin_nontemporal_store(w, dst + j);
        else dst[j] = w;
      }
    }
  }
  if (MODE == 0) {
    __shared__ sp_u32x4 red[256];
    red[threadIdx.x] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
      sp_u32x4 r = red[0];
      for (int t = 1; t < 256; ++t) r ^= red[t];
      dst[blockIdx.x] = r;
    }
  }
}

int stream_probe(int mode, bool nt, const void* src, void* dst, int64_t chunks, int blocks, hipStream_t s) {
  const double bytes = 16.0 * chunks * (mode == 2 ? 2.0 : 1.0);
  LaunchScope ls("stream_probe", s, 0.0, bytes);
  const sp_u32x4* in = static_cast<const sp_u32x4*>(src);
  sp_u32x4* out = static_cast<sp_u32x4*>(dst);
  const dim3 g(static_cast<unsigned>(blocks));
#define FF_STREAM(M)                                                                                       \
  if (nt) hipLaunchKernelGGL((stream_kernel<M, true>), g, dim3(256), 0, s, in, out, chunks);               \
  else hipLaunchKernelGGL((stream_kernel<M, false>), g, dim3(256), 0, s, in, out, chunks);
  if (mode == 0) { FF_STREAM(0) } else if (mode == 1) { FF_STREAM(1) } else { FF_STREAM(2) }
#undef FF_STREAM
  return ls.status();
}

int add_table(const void* table, int dtype, const float* e, float* out, int64_t B, int64_t n, hipStream_t s) {
  LaunchScope ls("add_table", s, 0.0, 8.0 * B * n);
  if (dtype == FF_BF16) hipLaunchKernelGGL(add_table_kernel<true>, dim3(blocks_for(B * n)), dim3(256), 0, s, table, e, out, B, n);
  else hipLaunchKernelGGL(add_table_kernel<false>, dim3(blocks_for(B * n)), dim3(256), 0, s, table, e, out, B, n);
  return ls.status();
}

}  // namespace ff
