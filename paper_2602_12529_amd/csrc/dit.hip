// DiT velocity forward v_theta(x_t, c, t): model handle, parameter table,
// workspace plan and the launch sequence of the dual-stream, single-stream and
// WAN blocks (block structure as documented in include/ff.h).
#include <cmath>
#include <cstring>
#include <string>
#include <memory>
#include <unordered_map>
#include <vector>

#include "ff_internal.h"

using namespace ff;

namespace {

struct TensorSpec {
  std::string name;
  int64_t s0, s1;   // s1 = 0 for 1-D
};

void lin(std::vector<TensorSpec>& t, const std::string& p, int64_t out, int64_t in) {
  t.push_back({p + ".w", out, in});
  t.push_back({p + ".b", out, 0});
}

std::vector<TensorSpec> tensor_table(const ff_dit_config& c) {
  std::vector<TensorSpec> t;
  const int64_t H = c.hidden, F = c.mlp_hidden, d = c.head_dim;
  const bool latent = c.io_mode == FF_IO_LATENT;
  if (c.model == FF_MODEL_MMDIT) {
    if (latent) {
      lin(t, "temb.fc1", H, 256);
      lin(t, "temb.fc2", H, H);
      if (c.pooled_dim) {
        lin(t, "pooled.fc1", H, c.pooled_dim);
        lin(t, "pooled.fc2", H, H);
      }
      lin(t, "x_in", H, c.in_channels);
      lin(t, "txt_in", H, c.txt_dim);
    }
    for (int i = 0; i < c.n_dual; ++i)
      for (const char* s : {"img", "txt"}) {
        std::string p = "dual." + std::to_string(i) + "." + s + ".";
        lin(t, p + "mod", 6 * H, H);
        lin(t, p + "qkv", 3 * H, H);
        t.push_back({p + "q_norm.w", d, 0});
        t.push_back({p + "k_norm.w", d, 0});
        lin(t, p + "o", H, H);
        lin(t, p + "mlp1", F, H);
        lin(t, p + "mlp2", H, F);
      }
    for (int j = 0; j < c.n_single; ++j) {
      std::string p = "single." + std::to_string(j) + ".";
      lin(t, p + "mod", 3 * H, H);
      lin(t, p + "lin1", 3 * H + F, H);
      t.push_back({p + "q_norm.w", d, 0});
      t.push_back({p + "k_norm.w", d, 0});
      lin(t, p + "lin2", H, H + F);
    }
    if (latent) {
      lin(t, "final.mod", 2 * H, H);
      lin(t, "final.proj", c.in_channels, H);
    }
  } else {
    if (latent) {
      lin(t, "temb.fc1", H, 256);
      lin(t, "temb.fc2", H, H);
      lin(t, "temb.proj", 6 * H, H);
      lin(t, "x_in", H, c.in_channels);
      lin(t, "txt_in.fc1", H, c.txt_dim);
      lin(t, "txt_in.fc2", H, H);
    }
    for (int i = 0; i < c.n_wan; ++i) {
      std::string p = "wan." + std::to_string(i) + ".";
      t.push_back({p + "mod", 6, H});
      lin(t, p + "sa.qkv", 3 * H, H);
      t.push_back({p + "sa.q_norm.w", H, 0});
      t.push_back({p + "sa.k_norm.w", H, 0});
      lin(t, p + "sa.o", H, H);
      t.push_back({p + "ca.norm.w", H, 0});
      t.push_back({p + "ca.norm.b", H, 0});
      lin(t, p + "ca.q", H, H);
      lin(t, p + "ca.kv", 2 * H, H);
      t.push_back({p + "ca.q_norm.w", H, 0});
      t.push_back({p + "ca.k_norm.w", H, 0});
      lin(t, p + "ca.o", H, H);
      lin(t, p + "ffn1", F, H);
      lin(t, p + "ffn2", H, F);
    }
    if (latent) {
      lin(t, "final.mod", 2 * H, H);
      lin(t, "final.proj", c.in_channels, H);
    }
  }
  return t;
}

// Size limits of a model and of a forward: they keep every tile count within a launch's 31-bit
// grid and every buffer size within 2^48 bytes (far beyond the models and batches in use).
constexpr int32_t kMaxBlocks = 4096, kMaxHidden = 1 << 16, kMaxHeads = 1024, kMaxMlp = 1 << 18, kMaxWidth = 1 << 16;
constexpr int64_t kMaxAxis = 1 << 20, kMaxRows = int64_t(1) << 27, kMaxTxt = 1 << 20;

int check_config(const ff_dit_config* c) {
  if (!c) return fail(FF_EINVAL, "ff_dit: null config");
  if (c->model != FF_MODEL_MMDIT && c->model != FF_MODEL_WAN) return fail(FF_EINVAL, "ff_dit: bad model %d", c->model);
  if (c->io_mode != FF_IO_LATENT && c->io_mode != FF_IO_HIDDEN) return fail(FF_EINVAL, "ff_dit: bad io_mode %d", c->io_mode);
  if (c->dtype != FF_F32 && c->dtype != FF_BF16) return fail(FF_EINVAL, "ff_dit: bad dtype %d", c->dtype);
  if (c->n_dual < 0 || c->n_single < 0 || c->n_wan < 0) return fail(FF_EINVAL, "ff_dit: negative block count");
  if (c->hidden <= 0 || c->heads <= 0 || c->head_dim <= 0 || c->mlp_hidden <= 0)
    return fail(FF_EINVAL, "ff_dit: non-positive size");
  if (c->n_dual > kMaxBlocks || c->n_single > kMaxBlocks || c->n_wan > kMaxBlocks)
    return fail(FF_EUNSUPPORTED, "ff_dit: more than %d blocks of one kind", kMaxBlocks);
  if (c->hidden > kMaxHidden || c->heads > kMaxHeads || c->mlp_hidden > kMaxMlp || c->in_channels > kMaxWidth ||
      c->txt_dim > kMaxWidth || c->pooled_dim > kMaxWidth)
    return fail(FF_EUNSUPPORTED, "ff_dit: a width above its limit (hidden %d, heads %d, MLP %d, other widths %d)",
                kMaxHidden, kMaxHeads, kMaxMlp, kMaxWidth);
  if (static_cast<int64_t>(c->heads) * c->head_dim != c->hidden)
    return fail(FF_EINVAL, "ff_dit: hidden %d != heads %d * head_dim %d", c->hidden, c->heads, c->head_dim);
  if (c->head_dim % 2) return fail(FF_EINVAL, "ff_dit: head_dim must be even");
  for (int a = 0; a < 3; ++a)
    if (c->rope_axes[a] < 0 || c->rope_axes[a] % 2) return fail(FF_EINVAL, "ff_dit: rope axis widths must be even and >= 0");
  if (static_cast<int64_t>(c->rope_axes[0]) + c->rope_axes[1] + c->rope_axes[2] != c->head_dim)
    return fail(FF_EINVAL, "ff_dit: rope axes must sum to head_dim");
  if (!(c->rope_theta > 0) || !(c->norm_eps > 0)) return fail(FF_EINVAL, "ff_dit: rope_theta and norm_eps must be > 0");
  if (c->norm_kind != FF_NORM_RMS && c->norm_kind != FF_NORM_LN) return fail(FF_EINVAL, "ff_dit: bad norm_kind");
  if (c->io_mode == FF_IO_LATENT && (c->in_channels <= 0 || c->txt_dim <= 0))
    return fail(FF_EINVAL, "ff_dit: latent mode needs in_channels and txt_dim");
  if (c->pooled_dim < 0) return fail(FF_EINVAL, "ff_dit: negative pooled_dim");
  if (c->dtype == FF_BF16) {
    if (c->head_dim != 128) return fail(FF_EUNSUPPORTED, "ff_dit: bf16 attention needs head_dim 128");
    const int64_t ks[] = {c->hidden, c->mlp_hidden, c->io_mode == FF_IO_LATENT ? c->in_channels : 64,
                          c->io_mode == FF_IO_LATENT ? c->txt_dim : 64};
    for (int64_t k : ks)
      if (k % 64) return fail(FF_EUNSUPPORTED, "ff_dit: bf16 layer widths must be multiples of 64 (got %lld)", (long long)k);
    if (c->pooled_dim % 8) return fail(FF_EUNSUPPORTED, "ff_dit: pooled_dim must be a multiple of 8");
  } else {
    if (c->head_dim > 64) return fail(FF_EUNSUPPORTED, "ff_dit: f32 attention needs head_dim <= 64");
    if (c->hidden % 8 || c->mlp_hidden % 8 || c->pooled_dim % 8)
      return fail(FF_EUNSUPPORTED, "ff_dit: f32 widths must be multiples of 8");
  }
  return FF_OK;
}

struct Lin {
  const void* w = nullptr;
  const void* b = nullptr;
};
struct Stream {
  Lin mod, qkv, o, mlp1, mlp2;
  const void* qn = nullptr;
  const void* kn = nullptr;
};
struct Single {
  Lin mod, lin1, lin2;
  const void* qn = nullptr;
  const void* kn = nullptr;
};
struct Wan {
  const void* mod = nullptr;            // E_block [6, H]
  Lin qkv, o, cq, ckv, co, ffn1, ffn2;
  const void* qn = nullptr;             // self-attention Q/K RMSNorm weights [H]
  const void* kn = nullptr;
  const void* can_w = nullptr;          // cross-attention query LayerNorm affine [H]
  const void* can_b = nullptr;
  const void* cqn = nullptr;            // cross-attention Q/K RMSNorm weights [H]
  const void* ckn = nullptr;
};

}  // namespace

struct ff_dit {
  ff_dit_config cfg;
  std::vector<const void*> ptr;
  Lin temb1, temb2, pooled1, pooled2, x_in, txt_in, final_mod, final_proj;
  Lin temb_proj, txt1, txt2;            // WAN: e(t) projection, text MLP
  std::vector<Stream> dual_img, dual_txt;
  std::vector<Single> single;
  std::vector<Wan> wan;
};

namespace {

// Workspace plan: byte offsets of every buffer of one forward.
struct Plan {
  int64_t B, Ni, Nt, N, P;
  size_t rope, temb_in, c, tmp, condB, cond32, mods, ximg, xtxt, joint, y, qkv, q, k, vt, o, u, txth;
  size_t e6, ctx1, ctxp, kvc, kc, vct, qd, sumsq, splitk, splitk_bytes, rowmap, block_mods, total;
};

Plan plan(const ff_dit& m, int64_t B, const int32_t grid[3], int64_t n_txt, int64_t n_prompts) {
  const ff_dit_config& c = m.cfg;
  Plan p{};
  p.B = B;
  p.Ni = static_cast<int64_t>(grid[0]) * grid[1] * grid[2];
  p.Nt = n_txt;
  p.N = p.Ni + p.Nt;
  p.P = n_prompts;
  const int64_t H = c.hidden, F = c.mlp_hidden;
  const size_t es = dtype_size(c.dtype);
  const bool latent = c.io_mode == FF_IO_LATENT;
  Carver cv(nullptr, 0);
  auto take = [&](size_t bytes) { void* q = cv.take(bytes); (void)q; return cv.off - bytes; };
  p.rope = take(static_cast<size_t>(p.Ni) * (c.head_dim / 2) * 8);
  p.temb_in = take(static_cast<size_t>(B) * 256 * 4);
  p.c = take(static_cast<size_t>(B) * H * 4);
  p.tmp = take(static_cast<size_t>(B) * H * 4);
  p.condB = take(static_cast<size_t>(B) * (c.pooled_dim > H ? c.pooled_dim : H) * es);
  p.cond32 = take(static_cast<size_t>(B) * (c.pooled_dim > H ? c.pooled_dim : H) * 4);
  p.mods = take(static_cast<size_t>(2) * B * 6 * H * 4);
  p.ximg = take(latent ? static_cast<size_t>(B) * p.Ni * H * es : 0);
  p.xtxt = take(static_cast<size_t>(B) * p.Nt * H * es);
  p.joint = take(c.n_single ? static_cast<size_t>(B) * p.N * H * es : 0);
  p.y = take(static_cast<size_t>(B) * p.N * H * es);
  p.qkv = take(static_cast<size_t>(B) * p.N * (3 * H + (c.n_single ? F : 0)) * es);
  p.q = take(static_cast<size_t>(B) * p.N * H * es);
  p.k = take(static_cast<size_t>(B) * p.N * H * es);
  p.vt = take(static_cast<size_t>(B) * p.N * H * es);
  p.o = take(static_cast<size_t>(B) * p.N * H * es);
  p.u = take(static_cast<size_t>(B) * (p.Ni + p.Nt) * F * es);
  p.txth = take(latent ? static_cast<size_t>(p.P) * p.Nt * H * es : 0);
  const bool wan = c.model == FF_MODEL_WAN;
  p.e6 = take(wan ? static_cast<size_t>(B) * 6 * H * 4 : 0);
  p.ctx1 = take(wan ? static_cast<size_t>(p.P) * p.Nt * H * es : 0);
  p.ctxp = take(wan ? static_cast<size_t>(p.P) * p.Nt * H * es : 0);
  p.kvc = take(wan ? static_cast<size_t>(B) * p.Nt * 2 * H * es : 0);
  p.kc = take(wan ? static_cast<size_t>(B) * p.Nt * H * es : 0);
  p.vct = take(wan ? static_cast<size_t>(B) * p.Nt * H * es : 0);
  p.qd = take(wan ? static_cast<size_t>(B) * p.Nt * H * es : 0);
  p.sumsq = take(wan ? static_cast<size_t>(B) * p.Ni * (2 * H / 64) * 4 : 0);
  p.splitk_bytes = c.dtype == FF_BF16 ? gemm_split_bytes() : 0;
  p.splitk = take(p.splitk_bytes);
  p.rowmap = take(static_cast<size_t>(row_classes_ints(B)) * 4);
  // every dual block's two [B, 6H] and every single block's [B, 3H] modulation vectors
  p.block_mods = take(static_cast<size_t>(B) * (c.n_dual * 12 + c.n_single * 3) * H * 4);
  p.total = round_up(cv.off, 256);
  return p;
}

inline char* at(void* ws, size_t off) { return static_cast<char*>(ws) + off; }

GemmArgs gemm_args(int dtype, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, Lin l, void* out,
                   int64_t ldo, int epi) {
  GemmArgs g{};
  g.dtype = dtype;
  g.M = M; g.N = N; g.K = K;
  g.A1 = A; g.lda1 = lda; g.K1 = K;
  g.A2 = nullptr; g.lda2 = 0;
  g.W = l.w; g.ldw = K;
  g.bias = l.b;
  g.out = out; g.ldo = ldo;
  g.epi = epi;
  g.gelu_from = 0;
  g.rows_per_sample = M;
  return g;
}

// The same, with the workspace's split-K scratch for the launch's last round.
GemmArgs gemm_args_ws(const Plan& p, void* ws, int dtype, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
                      Lin l, void* out, int64_t ldo, int epi) {
  GemmArgs g = gemm_args(dtype, M, N, K, A, lda, l, out, ldo, epi);
  if (p.splitk_bytes > 0 && dtype == FF_BF16) {
    g.split_ws = at(ws, p.splitk);
    g.split_bytes = p.splitk_bytes;
  }
  return g;
}

NormArgs norm_args(const ff_dit_config& c, int64_t rows, const void* x, void* y, const float* shift,
                   const float* scale, int64_t mod_ld, int64_t rows_per_sample) {
  NormArgs a{};
  a.dtype = c.dtype;
  a.rows = rows; a.H = c.hidden;
  a.x = x; a.ldx = c.hidden;
  a.y = y; a.ldy = c.hidden;
  a.norm_kind = c.norm_kind;
  a.eps = static_cast<float>(c.norm_eps);
  a.shift = shift; a.scale = scale; a.mod_ld = mod_ld;
  a.w = nullptr; a.bias = nullptr;
  a.rows_per_sample = rows_per_sample;
  return a;
}

SkinnyArgs skinny_args(int dtype, int64_t B, int64_t N, int64_t K, const float* in, int act_in, Lin l, float* out,
                       int accumulate = 0, int act_out = ACT_NONE, const int32_t* rowmap = nullptr) {
  SkinnyArgs s{};
  s.rowmap = rowmap;
  s.dtype = dtype;
  s.B = B; s.N = N; s.K = K;
  s.in = in; s.ldi = K; s.act_in = act_in;
  s.W = l.w; s.bias = l.b;
  s.out = out; s.ldo = N;
  s.accumulate = accumulate;
  s.act_out = act_out;
  return s;
}

// QK norm + RoPE + relayout for one stream's rows: source row of token i of sample b is
// b * src_rows + src_off + i.
QkvArgs qkv_args(const ff_dit_config& c, const Plan& p, void* ws, const void* qkv_base, int64_t ld, int64_t src_rows,
                 int64_t src_off, int64_t n_tok, int64_t tok_offset, const void* qn, const void* kn, bool rope) {
  const size_t es = dtype_size(c.dtype);
  const char* base = static_cast<const char*>(qkv_base) + src_off * ld * es;
  QkvArgs a{};
  a.dtype = c.dtype;
  a.B = p.B; a.n_tok = n_tok; a.tok_offset = tok_offset; a.n_joint = p.N;
  a.heads = c.heads; a.d = c.head_dim;
  a.q = base; a.k = base + c.hidden * es; a.v = base + 2 * c.hidden * es;
  a.ld = ld;
  a.q_w = qn; a.k_w = kn;
  a.full_width_norm = 0;
  a.apply_norm = 1;
  a.eps = static_cast<float>(c.norm_eps);
  a.rope = rope ? reinterpret_cast<const float2*>(at(ws, p.rope)) : nullptr;
  a.Q = at(ws, p.q); a.Kd = at(ws, p.k); a.Vt = at(ws, p.vt);
  a.v_transposed = c.dtype == FF_BF16;
  a.src_rows = src_rows;
  return a;
}

int qkv_stream(const ff_dit_config& c, const Plan& p, void* ws, const void* qkv_base, int64_t ld, int64_t src_rows,
               int64_t src_off, int64_t n_tok, int64_t tok_offset, const void* qn, const void* kn, bool rope,
               hipStream_t s) {
  return qk_norm_rope(qkv_args(c, p, ws, qkv_base, ld, src_rows, src_off, n_tok, tok_offset, qn, kn, rope), s);
}

int attention_joint(const ff_dit_config& c, const Plan& p, void* ws, void* out_txt, void* out_img, hipStream_t s) {
  AttnArgs a{};
  a.dtype = c.dtype;
  a.B = p.B; a.heads = c.heads; a.d = c.head_dim;
  a.n_q = p.N; a.n_kv = p.N;
  a.Q = at(ws, p.q); a.K = at(ws, p.k); a.Vt = at(ws, p.vt);
  a.out0 = out_txt; a.out1 = out_img; a.split = p.Nt; a.ldo = c.hidden;
  a.scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(c.head_dim)));
  return attention(a, s);
}

// Where block_modulations leaves the modulation vectors: dual block i, stream k (0 text, 1 image)
// [B, 6H]; then single block j [B, 3H].
float* dual_mods(const Plan& p, void* ws, int64_t H, int i, int k) {
  return reinterpret_cast<float*>(at(ws, p.block_mods)) + (2 * static_cast<int64_t>(i) + k) * p.B * 6 * H;
}
float* single_mods(const ff_dit& m, const Plan& p, void* ws, int64_t H, int j) {
  return reinterpret_cast<float*>(at(ws, p.block_mods)) + m.cfg.n_dual * 2 * p.B * 6 * H + static_cast<int64_t>(j) * p.B * 3 * H;
}

// All blocks' adaLN modulation vectors W_mod SiLU(c) + b from the same c, one row per class of
// equal conditioning rows, in as few launches as there are groups of 40 weight matrices: one long
// weight stream instead of a short launch per block and stream.
int block_modulations(const ff_dit& m, const Plan& p, void* ws, const float* c32, hipStream_t s) {
  const ff_dit_config& c = m.cfg;
  const int64_t H = c.hidden;
  std::vector<SkinnySeg> segs;
  segs.reserve(2 * c.n_dual + c.n_single);
  for (int i = 0; i < c.n_dual; ++i) {
    segs.push_back({m.dual_txt[i].mod.w, m.dual_txt[i].mod.b, dual_mods(p, ws, H, i, 0), 6 * H});
    segs.push_back({m.dual_img[i].mod.w, m.dual_img[i].mod.b, dual_mods(p, ws, H, i, 1), 6 * H});
  }
  for (int j = 0; j < c.n_single; ++j) segs.push_back({m.single[j].mod.w, m.single[j].mod.b, single_mods(m, p, ws, H, j), 3 * H});
  SkinnyArgs a = skinny_args(c.dtype, p.B, 0, H, c32, ACT_SILU, Lin{}, nullptr, 0, ACT_NONE,
                             reinterpret_cast<const int32_t*>(at(ws, p.rowmap)));
  return skinny_linear_multi(a, segs.data(), static_cast<int>(segs.size()), s);
}

// One dual-stream block.  cur[s] is the stream's current residual (input of the block);
// dst[s] receives the updated residual (may equal cur[s]).
int dual_block(const ff_dit& m, const Plan& p, void* ws, int i, const float* c32, const void* cur[2], void* dst[2],
               hipStream_t s) {
  const ff_dit_config& c = m.cfg;
  const int64_t H = c.hidden, F = c.mlp_hidden;
  const size_t es = dtype_size(c.dtype);
  const Stream* st[2] = {&m.dual_txt[i], &m.dual_img[i]};
  const int64_t rows[2] = {p.B * p.Nt, p.B * p.Ni};
  const int64_t ntok[2] = {p.Nt, p.Ni};
  const int64_t y_off[2] = {0, p.B * p.Nt * H};    // Y / O rows: txt rows first, then img rows
  float* mods[2] = {dual_mods(p, ws, H, i, 0), dual_mods(p, ws, H, i, 1)};   // computed by block_modulations
  char* Y = at(ws, p.y);
  char* O = at(ws, p.o);
  char* QKV = at(ws, p.qkv);
  char* qkv_k[2] = {QKV, QKV + p.B * p.Nt * 3 * H * es};
  char* U[2] = {at(ws, p.u), at(ws, p.u) + p.B * p.Nt * F * es};
  for (int k = 0; k < 2; ++k) {
    FF_TRY(norm_modulate(norm_args(c, rows[k], cur[k], Y + y_off[k] * es, mods[k], mods[k] + H, 6 * H, ntok[k]), s));
  }
  // QKV projections of both streams; the QK norm, rotation and relayout run in the GEMM epilogue
  // when the shapes allow (gemm2 falls back to a second pass otherwise).
  QkvArgs qa[2];
  GemmArgs gq[2];
  for (int k = 0; k < 2; ++k) {
    qa[k] = qkv_args(c, p, ws, qkv_k[k], 3 * H, ntok[k], 0, ntok[k], k == 0 ? 0 : p.Nt, st[k]->qn, st[k]->kn, k == 1);
    gq[k] = gemm_args_ws(p, ws, c.dtype, rows[k], 3 * H, H, Y + y_off[k] * es, H, st[k]->qkv, qkv_k[k], 3 * H, EPI_QKV);
    gq[k].qkv = &qa[k];
  }
  FF_TRY(gemm2(gq[0], gq[1], s));
  FF_TRY(attention_joint(c, p, ws, O, O + p.B * p.Nt * H * es, s));
  GemmArgs go[2], g1[2], g2[2];
  for (int k = 0; k < 2; ++k) {
    go[k] = gemm_args_ws(p, ws, c.dtype, rows[k], H, H, O + y_off[k] * es, H, st[k]->o, dst[k], H, EPI_GATED);
    go[k].gate = mods[k] + 2 * H; go[k].gate_ld = 6 * H;
    go[k].resid = cur[k]; go[k].ldr = H;
    go[k].rows_per_sample = ntok[k];
  }
  FF_TRY(gemm2(go[0], go[1], s));
  for (int k = 0; k < 2; ++k) {
    FF_TRY(norm_modulate(norm_args(c, rows[k], dst[k], Y + y_off[k] * es, mods[k] + 3 * H, mods[k] + 4 * H, 6 * H, ntok[k]), s));
    g1[k] = gemm_args_ws(p, ws, c.dtype, rows[k], F, H, Y + y_off[k] * es, H, st[k]->mlp1, U[k], F, EPI_GELU);
    g2[k] = gemm_args_ws(p, ws, c.dtype, rows[k], H, F, U[k], F, st[k]->mlp2, dst[k], H, EPI_GATED);
    g2[k].gate = mods[k] + 5 * H; g2[k].gate_ld = 6 * H;
    g2[k].resid = dst[k]; g2[k].ldr = H;
    g2[k].rows_per_sample = ntok[k];
  }
  FF_TRY(gemm2(g1[0], g1[1], s));
  FF_TRY(gemm2(g2[0], g2[1], s));
  return FF_OK;
}

// One single-stream block on the joint residual X [B, N, H] (txt rows first), in place.
int single_block(const ff_dit& m, const Plan& p, void* ws, int j, const float* c32, void* X, hipStream_t s) {
  const ff_dit_config& c = m.cfg;
  const int64_t H = c.hidden, F = c.mlp_hidden, W1 = 3 * H + F;
  const size_t es = dtype_size(c.dtype);
  const Single& sb = m.single[j];
  float* mods = single_mods(m, p, ws, H, j);   // computed by block_modulations
  const int64_t rows = p.B * p.N;
  char* Y = at(ws, p.y);
  char* H1 = at(ws, p.qkv);
  char* O = at(ws, p.o);
  FF_TRY(norm_modulate(norm_args(c, rows, X, Y, mods, mods + H, 3 * H, p.N), s));
  // [Q | K | V | MLP input] in one GEMM: Q, K, V of the joint sequence go to the attention layout
  // (text tokens unrotated, image tokens rotated by their grid position), GELU from column 3H.
  QkvArgs qa = qkv_args(c, p, ws, H1, W1, p.N, 0, p.N, 0, sb.qn, sb.kn, true);
  qa.rope_from = p.Nt;
  GemmArgs g1 = gemm_args_ws(p, ws, c.dtype, rows, W1, H, Y, H, sb.lin1, H1, W1, EPI_QKV);
  g1.gelu_from = 3 * H;
  g1.qkv = &qa;
  FF_TRY(gemm(g1, s));
  AttnArgs a{};
  a.dtype = c.dtype;
  a.B = p.B; a.heads = c.heads; a.d = c.head_dim;
  a.n_q = p.N; a.n_kv = p.N;
  a.Q = at(ws, p.q); a.K = at(ws, p.k); a.Vt = at(ws, p.vt);
  a.out0 = O; a.out1 = O; a.split = p.N; a.ldo = H;
  a.scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(c.head_dim)));
  FF_TRY(attention(a, s));
  GemmArgs g2 = gemm_args_ws(p, ws, c.dtype, rows, H, H + F, O, H, sb.lin2, X, H, EPI_GATED);
  g2.K1 = H;
  g2.A2 = H1 + 3 * H * es; g2.lda2 = W1;
  g2.gate = mods + 2 * H; g2.gate_ld = 3 * H;
  g2.resid = X; g2.ldr = H;
  g2.rows_per_sample = p.N;
  return gemm(g2, s);
}

// In-place RMSNorm * w over rows of width H with row stride ld (full-width QK norm).
int rms_rows(const ff_dit_config& c, void* x, int64_t rows, int64_t ld, const void* w, hipStream_t s) {
  NormArgs a{};
  a.dtype = c.dtype;
  a.rows = rows; a.H = c.hidden;
  a.x = x; a.ldx = ld; a.y = x; a.ldy = ld;
  a.norm_kind = FF_NORM_RMS;
  a.eps = static_cast<float>(c.norm_eps);
  a.shift = nullptr; a.scale = nullptr; a.mod_ld = 0;
  a.w = w; a.bias = nullptr;
  a.rows_per_sample = rows;
  return norm_modulate(a, s);
}

// Relayout (no norm, optional RoPE) of packed Q|K|V rows into the attention layout.
int relayout(const ff_dit_config& c, const Plan& p, const void* q, const void* k, const void* v, int64_t ld,
             int64_t n_tok, const float2* rope, void* Q, void* K, void* Vt, hipStream_t s) {
  QkvArgs a{};
  a.dtype = c.dtype;
  a.B = p.B; a.n_tok = n_tok; a.tok_offset = 0; a.n_joint = n_tok; a.src_rows = n_tok;
  a.heads = c.heads; a.d = c.head_dim;
  a.q = q; a.k = k; a.v = v; a.ld = ld;
  a.q_w = nullptr; a.k_w = nullptr;
  a.full_width_norm = 0; a.apply_norm = 0;
  a.eps = static_cast<float>(c.norm_eps);
  a.rope = rope;
  a.Q = Q; a.Kd = K; a.Vt = Vt;
  a.v_transposed = c.dtype == FF_BF16;
  return qk_norm_rope(a, s);
}

// Block i's cross-attention keys and values from the text context ctx [B*N_txt, H]: one GEMM to
// [K | V], the RMSNorm of K over all of H, and the relayout to K [B, h, N_txt, d] and V^T.
int wan_cross_kv(const ff_dit& m, const Plan& p, void* ws, int i, const void* ctx, void* K, void* Vt, hipStream_t s);

// One WAN block on X [B*N_img, H] in place; mods [B, 6H].  The cross-attention reads K / V^T from
// ctx_k / ctx_vt when given (prepared once per rollout), else computes them from ctx [B*N_txt, H].
int wan_block(const ff_dit& m, const Plan& p, void* ws, int i, const void* ctx, const void* ctx_k,
              const void* ctx_vt, void* X, hipStream_t s) {
  const ff_dit_config& c = m.cfg;
  const int64_t H = c.hidden, F = c.mlp_hidden;
  const size_t es = dtype_size(c.dtype);
  const Wan& wb = m.wan[i];
  const int64_t rows = p.B * p.Ni, crow = p.B * p.Nt;
  float* mods = reinterpret_cast<float*>(at(ws, p.mods));
  const float* e6 = reinterpret_cast<const float*>(at(ws, p.e6));
  char* Y = at(ws, p.y);
  char* QKV = at(ws, p.qkv);
  char* O = at(ws, p.o);
  const float scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(c.head_dim)));
  FF_TRY(add_table(wb.mod, c.dtype, e6, mods, p.B, 6 * H, s));
  // self-attention
  FF_TRY(norm_modulate(norm_args(c, rows, X, Y, mods, mods + H, 6 * H, p.Ni), s));
  // Q, K with their RMSNorm over all of H, rotated, and V: the projection's epilogue leaves each
  // token's partial sums of q^2 and k^2 per 64 columns, and one relayout pass normalises, rotates
  // and moves Q, K, V^T to the attention layout.  Shapes the tile kernel does not take use the
  // two in-place norm passes and a plain relayout.
  GemmArgs gq = gemm_args_ws(p, ws, c.dtype, rows, 3 * H, H, Y, H, wb.qkv, QKV, 3 * H, EPI_SUMSQ);
  gq.sumsq = reinterpret_cast<float*>(at(ws, p.sumsq));
  gq.sumsq_w = H;
  const float2* rope = reinterpret_cast<const float2*>(at(ws, p.rope));
  QkvArgs qa{};
  if (c.head_dim == 128 && gemm_sumsq_ok(gq)) {
    FF_TRY(gemm(gq, s));
    qa.dtype = c.dtype;
    qa.B = p.B; qa.n_tok = p.Ni; qa.tok_offset = 0; qa.n_joint = p.Ni; qa.src_rows = p.Ni;
    qa.heads = c.heads; qa.d = c.head_dim;
    qa.q = QKV; qa.k = QKV + H * es; qa.v = QKV + 2 * H * es; qa.ld = 3 * H;
    qa.q_w = wb.qn; qa.k_w = wb.kn;
    qa.full_width_norm = 1; qa.apply_norm = 1;
    qa.eps = static_cast<float>(c.norm_eps);
    qa.rope = rope;
    qa.Q = at(ws, p.q); qa.Kd = at(ws, p.k); qa.Vt = at(ws, p.vt);
    qa.v_transposed = 1;
    qa.sumsq = gq.sumsq;
    qa.sumsq_parts = 2 * H / 64;
    FF_TRY(qk_norm_rope(qa, s));
  } else {
    FF_TRY(gemm(gemm_args_ws(p, ws, c.dtype, rows, 3 * H, H, Y, H, wb.qkv, QKV, 3 * H, EPI_NONE), s));
    FF_TRY(rms_rows(c, QKV, rows, 3 * H, wb.qn, s));
    FF_TRY(rms_rows(c, QKV + H * es, rows, 3 * H, wb.kn, s));
    FF_TRY(relayout(c, p, QKV, QKV + H * es, QKV + 2 * H * es, 3 * H, p.Ni, rope, at(ws, p.q), at(ws, p.k),
                    at(ws, p.vt), s));
  }
  {
    AttnArgs a{};
    a.dtype = c.dtype;
    a.B = p.B; a.heads = c.heads; a.d = c.head_dim;
    a.n_q = p.Ni; a.n_kv = p.Ni;
    a.Q = at(ws, p.q); a.K = at(ws, p.k); a.Vt = at(ws, p.vt);
    a.out0 = O; a.out1 = O; a.split = p.Ni; a.ldo = H;
    a.scale = scale;
    FF_TRY(attention(a, s));
  }
  GemmArgs go = gemm_args_ws(p, ws, c.dtype, rows, H, H, O, H, wb.o, X, H, EPI_GATED);
  go.gate = mods + 2 * H; go.gate_ld = 6 * H; go.resid = X; go.ldr = H; go.rows_per_sample = p.Ni;
  FF_TRY(gemm(go, s));
  // cross-attention to the text context (K/V from ctx; Q read token-major)
  {
    NormArgs na = norm_args(c, rows, X, Y, nullptr, nullptr, 0, p.Ni);
    na.norm_kind = FF_NORM_LN;
    na.w = wb.can_w; na.bias = wb.can_b;
    FF_TRY(norm_modulate(na, s));
  }
  FF_TRY(gemm(gemm_args_ws(p, ws, c.dtype, rows, H, H, Y, H, wb.cq, QKV, H, EPI_NONE), s));
  FF_TRY(rms_rows(c, QKV, rows, H, wb.cqn, s));
  if (!ctx_k) {
    FF_TRY(wan_cross_kv(m, p, ws, i, ctx, at(ws, p.kc), at(ws, p.vct), s));
    ctx_k = at(ws, p.kc);
    ctx_vt = at(ws, p.vct);
  }
  {
    AttnArgs a{};
    a.dtype = c.dtype;
    a.B = p.B; a.heads = c.heads; a.d = c.head_dim;
    a.n_q = p.Ni; a.n_kv = p.Nt;
    a.Q = QKV; a.K = ctx_k; a.Vt = ctx_vt;
    a.q_bs = p.Ni * H; a.q_hs = c.head_dim; a.q_rs = H;
    a.out0 = O; a.out1 = O; a.split = p.Ni; a.ldo = H;
    a.scale = scale;
    FF_TRY(attention(a, s));
  }
  GemmArgs gc = gemm_args_ws(p, ws, c.dtype, rows, H, H, O, H, wb.co, X, H, EPI_GATED);
  gc.gate = nullptr; gc.resid = X; gc.ldr = H; gc.rows_per_sample = p.Ni;
  FF_TRY(gemm(gc, s));
  // FFN
  FF_TRY(norm_modulate(norm_args(c, rows, X, Y, mods + 3 * H, mods + 4 * H, 6 * H, p.Ni), s));
  char* U = at(ws, p.u);
  FF_TRY(gemm(gemm_args_ws(p, ws, c.dtype, rows, F, H, Y, H, wb.ffn1, U, F, EPI_GELU), s));
  GemmArgs g2 = gemm_args_ws(p, ws, c.dtype, rows, H, F, U, F, wb.ffn2, X, H, EPI_GATED);
  g2.gate = mods + 5 * H; g2.gate_ld = 6 * H; g2.resid = X; g2.ldr = H; g2.rows_per_sample = p.Ni;
  return gemm(g2, s);
}

int wan_cross_kv(const ff_dit& m, const Plan& p, void* ws, int i, const void* ctx, void* K, void* Vt, hipStream_t s) {
  const ff_dit_config& c = m.cfg;
  const int64_t H = c.hidden;
  const size_t es = dtype_size(c.dtype);
  const Wan& wb = m.wan[i];
  const int64_t crow = p.B * p.Nt;
  char* KV = at(ws, p.kvc);
  FF_TRY(gemm(gemm_args_ws(p, ws, c.dtype, crow, 2 * H, H, ctx, H, wb.ckv, KV, 2 * H, EPI_NONE), s));
  FF_TRY(rms_rows(c, KV, crow, 2 * H, wb.ckn, s));
  return relayout(c, p, KV, KV, KV + H * es, 2 * H, p.Nt, nullptr, at(ws, p.qd), K, Vt, s);
}

// Bytes of one block's prepared cross-attention K and V^T, and the text context of a WAN forward:
// the embedding MLP of the prompts' text and the per-sample gather, into the workspace's xtxt.
size_t wan_kv_block_bytes(const ff_dit_config& c, int64_t B, int64_t n_txt) {
  return round_up(static_cast<size_t>(B) * n_txt * c.hidden * dtype_size(c.dtype), 256);
}

int wan_text_context(const ff_dit& m, const Plan& p, const void* txt, const int32_t* txt_index, void* ws,
                     hipStream_t s) {
  const ff_dit_config& c = m.cfg;
  const int64_t H = c.hidden;
  char* c1 = at(ws, p.ctx1);
  char* cp = at(ws, p.ctxp);
  FF_TRY(gemm(gemm_args_ws(p, ws, c.dtype, p.P * p.Nt, H, c.txt_dim, txt, c.txt_dim, m.txt1, c1, H, EPI_GELU), s));
  FF_TRY(gemm(gemm_args_ws(p, ws, c.dtype, p.P * p.Nt, H, H, c1, H, m.txt2, cp, H, EPI_NONE), s));
  return gather_rows(c.dtype, cp, txt_index, p.P, at(ws, p.xtxt), p.B, p.Nt, H, s);
}

// store: the prepared per-block cross-attention K / V^T (then txt is not read), or null.
int forward_wan(const ff_dit& m, const Plan& p, const void* x, const void* txt, const int32_t* txt_index,
                const float* t, const int32_t grid[3], void* v_out, void* ws, const char* store, hipStream_t s) {
  const ff_dit_config& c = m.cfg;
  const int64_t H = c.hidden;
  float* temb = reinterpret_cast<float*>(at(ws, p.c));
  float* tmp = reinterpret_cast<float*>(at(ws, p.tmp));
  float* te = reinterpret_cast<float*>(at(ws, p.temb_in));
  FF_TRY(rope_table(reinterpret_cast<float2*>(at(ws, p.rope)), grid, c.head_dim, c.rope_axes, c.rope_theta, s));
  FF_TRY(timestep_sinusoid(t, te, p.B, s));
  FF_TRY(skinny_linear(skinny_args(c.dtype, p.B, H, 256, te, ACT_NONE, m.temb1, tmp), s));
  FF_TRY(skinny_linear(skinny_args(c.dtype, p.B, H, H, tmp, ACT_SILU, m.temb2, temb), s));
  FF_TRY(skinny_linear(skinny_args(c.dtype, p.B, 6 * H, H, temb, ACT_SILU, m.temb_proj, reinterpret_cast<float*>(at(ws, p.e6))), s));
  char* ctx = at(ws, p.xtxt);
  if (!store) FF_TRY(wan_text_context(m, p, txt, txt_index, ws, s));
  char* X = at(ws, p.ximg);
  FF_TRY(gemm(gemm_args_ws(p, ws, c.dtype, p.B * p.Ni, H, c.in_channels, x, c.in_channels, m.x_in, X, H, EPI_NONE), s));
  const size_t kvb = wan_kv_block_bytes(c, p.B, p.Nt);
  for (int i = 0; i < c.n_wan; ++i) {
    const char* k = store ? store + 2 * i * kvb : nullptr;
    FF_TRY(wan_block(m, p, ws, i, ctx, k, store ? k + kvb : nullptr, X, s));
  }
  float* mods = reinterpret_cast<float*>(at(ws, p.mods));
  FF_TRY(skinny_linear(skinny_args(c.dtype, p.B, 2 * H, H, temb, ACT_SILU, m.final_mod, mods), s));
  char* Y = at(ws, p.y);
  FF_TRY(norm_modulate(norm_args(c, p.B * p.Ni, X, Y, mods, mods + H, 2 * H, p.Ni), s));
  return gemm(gemm_args_ws(p, ws, c.dtype, p.B * p.Ni, c.in_channels, H, Y, H, m.final_proj, v_out, c.in_channels, EPI_NONE), s);
}

int forward_mmdit(const ff_dit& m, const Plan& p, const void* x, const void* txt, const int32_t* txt_index,
                  const void* cond, const float* t, const int32_t grid[3], void* v_out, void* txt_out, void* ws,
                  hipStream_t s) {
  const ff_dit_config& c = m.cfg;
  const int64_t H = c.hidden;
  const size_t es = dtype_size(c.dtype);
  const bool latent = c.io_mode == FF_IO_LATENT;
  float* c32 = reinterpret_cast<float*>(at(ws, p.c));
  FF_TRY(rope_table(reinterpret_cast<float2*>(at(ws, p.rope)), grid, c.head_dim, c.rope_axes, c.rope_theta, s));

  const void* cur[2];
  void* dst[2];
  if (latent) {
    float* te = reinterpret_cast<float*>(at(ws, p.temb_in));
    float* tmp = reinterpret_cast<float*>(at(ws, p.tmp));
    FF_TRY(timestep_sinusoid(t, te, p.B, s));
    FF_TRY(skinny_linear(skinny_args(c.dtype, p.B, H, 256, te, ACT_NONE, m.temb1, tmp), s));
    FF_TRY(skinny_linear(skinny_args(c.dtype, p.B, H, H, tmp, ACT_SILU, m.temb2, c32), s));
    if (c.pooled_dim) {
      float* cond32 = reinterpret_cast<float*>(at(ws, p.cond32));
      FF_TRY(gather_rows(c.dtype, cond, txt_index, p.P, at(ws, p.condB), p.B, 1, c.pooled_dim, s));
      FF_TRY(cast_to_f32(c.dtype, at(ws, p.condB), cond32, p.B * c.pooled_dim, s));
      FF_TRY(skinny_linear(skinny_args(c.dtype, p.B, H, c.pooled_dim, cond32, ACT_NONE, m.pooled1, tmp), s));
      FF_TRY(skinny_linear(skinny_args(c.dtype, p.B, H, H, tmp, ACT_SILU, m.pooled2, c32, 1), s));
    }
    char* ximg = at(ws, p.ximg);
    FF_TRY(gemm(gemm_args_ws(p, ws, c.dtype, p.B * p.Ni, H, c.in_channels, x, c.in_channels, m.x_in, ximg, H, EPI_NONE), s));
    char* txth = at(ws, p.txth);
    FF_TRY(gemm(gemm_args_ws(p, ws, c.dtype, p.P * p.Nt, H, c.txt_dim, txt, c.txt_dim, m.txt_in, txth, H, EPI_NONE), s));
    FF_TRY(gather_rows(c.dtype, txth, txt_index, p.P, at(ws, p.xtxt), p.B, p.Nt, H, s));
    cur[0] = at(ws, p.xtxt);
    cur[1] = ximg;
    dst[0] = at(ws, p.xtxt);
    dst[1] = ximg;
  } else {
    FF_TRY(cast_to_f32(c.dtype, cond, c32, p.B * H, s));
    cur[0] = txt;
    cur[1] = x;
    dst[0] = txt_out ? txt_out : static_cast<void*>(at(ws, p.xtxt));
    dst[1] = v_out;
  }

  // Samples at the same time step with the same prompt share c, hence every modulation vector:
  // the block GEMVs compute each distinct row of c once.
  FF_TRY(row_classes(c32, p.B, H, reinterpret_cast<int32_t*>(at(ws, p.rowmap)), s));
  FF_TRY(block_modulations(m, p, ws, c32, s));
  for (int i = 0; i < c.n_dual; ++i) {
    FF_TRY(dual_block(m, p, ws, i, c32, cur, dst, s));
    cur[0] = dst[0];
    cur[1] = dst[1];
  }
  if (c.n_single) {
    char* X = at(ws, p.joint);
    const size_t row = static_cast<size_t>(H) * es;
    FF_CHECK_HIP(hipMemcpy2DAsync(X, p.N * row, cur[0], p.Nt * row, p.Nt * row, p.B, hipMemcpyDeviceToDevice, s), "copy txt->joint");
    FF_CHECK_HIP(hipMemcpy2DAsync(X + p.Nt * row, p.N * row, cur[1], p.Ni * row, p.Ni * row, p.B, hipMemcpyDeviceToDevice, s), "copy img->joint");
    for (int j = 0; j < c.n_single; ++j) FF_TRY(single_block(m, p, ws, j, c32, X, s));
    void* img_dst = latent ? static_cast<void*>(at(ws, p.ximg)) : v_out;
    FF_CHECK_HIP(hipMemcpy2DAsync(img_dst, p.Ni * row, X + p.Nt * row, p.N * row, p.Ni * row, p.B, hipMemcpyDeviceToDevice, s), "copy joint->img");
    if (!latent && txt_out)
      FF_CHECK_HIP(hipMemcpy2DAsync(txt_out, p.Nt * row, X, p.N * row, p.Nt * row, p.B, hipMemcpyDeviceToDevice, s), "copy joint->txt");
    cur[1] = img_dst;
  } else if (!latent && c.n_dual == 0) {
    // No blocks: outputs are the inputs.
    FF_CHECK_HIP(hipMemcpyAsync(v_out, x, static_cast<size_t>(p.B) * p.Ni * H * es, hipMemcpyDeviceToDevice, s), "copy x");
    if (txt_out)
      FF_CHECK_HIP(hipMemcpyAsync(txt_out, txt, static_cast<size_t>(p.B) * p.Nt * H * es, hipMemcpyDeviceToDevice, s), "copy txt");
  }

  if (latent) {
    float* mods = reinterpret_cast<float*>(at(ws, p.mods));
    FF_TRY(skinny_linear(skinny_args(c.dtype, p.B, 2 * H, H, c32, ACT_SILU, m.final_mod, mods, 0, ACT_NONE,
                                     reinterpret_cast<const int32_t*>(at(ws, p.rowmap))), s));
    char* Y = at(ws, p.y);
    FF_TRY(norm_modulate(norm_args(c, p.B * p.Ni, cur[1], Y, mods, mods + H, 2 * H, p.Ni), s));
    FF_TRY(gemm(gemm_args_ws(p, ws, c.dtype, p.B * p.Ni, c.in_channels, H, Y, H, m.final_proj, v_out, c.in_channels, EPI_NONE), s));
  }
  return FF_OK;
}

// Runs an entry point's body so that no C++ exception (a failed host allocation) leaves the C ABI.
template <typename F>
int guarded(const char* fn, F&& body) {
  try {
    return body();
  } catch (const std::bad_alloc&) {
    return fail(FF_EUNSUPPORTED, "%s: out of host memory", fn);
  } catch (...) {
    return fail(FF_EINVAL, "%s: internal error", fn);
  }
}

}  // namespace

extern "C" {

int ff_dit_num_tensors(const ff_dit_config* cfg, int64_t* n) {
  return guarded("ff_dit_num_tensors", [&]() -> int {
    FF_TRY(check_config(cfg));
    if (!n) return fail(FF_EINVAL, "ff_dit_num_tensors: null output");
    *n = static_cast<int64_t>(tensor_table(*cfg).size());
    return FF_OK;
  });
}

int ff_dit_tensor_info(const ff_dit_config* cfg, int64_t i, char* name, size_t name_cap, int64_t* shape0,
                       int64_t* shape1) {
  return guarded("ff_dit_tensor_info", [&]() -> int {
    FF_TRY(check_config(cfg));
    std::vector<TensorSpec> t = tensor_table(*cfg);
    if (i < 0 || i >= static_cast<int64_t>(t.size())) return fail(FF_EINVAL, "ff_dit_tensor_info: index %lld out of range", (long long)i);
    if (name) {
      if (name_cap < t[i].name.size() + 1) return fail(FF_EINVAL, "ff_dit_tensor_info: name buffer too small");
      memcpy(name, t[i].name.c_str(), t[i].name.size() + 1);
    }
    if (shape0) *shape0 = t[i].s0;
    if (shape1) *shape1 = t[i].s1;
    return FF_OK;
  });
}

int ff_dit_create(const ff_dit_config* cfg, const void* const* tensors, int64_t n_tensors, ff_dit** out) {
  return guarded("ff_dit_create", [&]() -> int {
    FF_TRY(check_config(cfg));
    if (cfg->model == FF_MODEL_WAN && cfg->io_mode != FF_IO_LATENT)
      return fail(FF_EUNSUPPORTED, "ff_dit_create: the WAN model runs in latent mode only");
    if (!out) return fail(FF_EINVAL, "ff_dit_create: null output");
    *out = nullptr;
    std::vector<TensorSpec> t = tensor_table(*cfg);
    if (n_tensors != static_cast<int64_t>(t.size()))
      return fail(FF_EINVAL, "ff_dit_create: %lld tensors given, %zu expected", (long long)n_tensors, t.size());
    if (!tensors) return fail(FF_EINVAL, "ff_dit_create: null tensor array");
    std::unordered_map<std::string, const void*> by;
    for (size_t i = 0; i < t.size(); ++i) {
      if (!tensors[i]) return fail(FF_EINVAL, "ff_dit_create: tensor %zu (%s) is null", i, t[i].name.c_str());
      if (!aligned16(tensors[i])) return fail(FF_EINVAL, "ff_dit_create: tensor %s not 16-byte aligned", t[i].name.c_str());
      by[t[i].name] = tensors[i];
    }
    std::unique_ptr<ff_dit> m(new ff_dit());
    m->cfg = *cfg;
    m->ptr.assign(tensors, tensors + n_tensors);
    auto L = [&](const std::string& p) { Lin l; l.w = by[p + ".w"]; l.b = by[p + ".b"]; return l; };
    if (cfg->io_mode == FF_IO_LATENT) {
      m->temb1 = L("temb.fc1");
      m->temb2 = L("temb.fc2");
      if (cfg->model == FF_MODEL_MMDIT) {
        if (cfg->pooled_dim) { m->pooled1 = L("pooled.fc1"); m->pooled2 = L("pooled.fc2"); }
        m->txt_in = L("txt_in");
      } else {
        m->temb_proj = L("temb.proj");
        m->txt1 = L("txt_in.fc1");
        m->txt2 = L("txt_in.fc2");
      }
      m->x_in = L("x_in");
      m->final_mod = L("final.mod");
      m->final_proj = L("final.proj");
    }
    for (int i = 0; i < (cfg->model == FF_MODEL_WAN ? cfg->n_wan : 0); ++i) {
      std::string p = "wan." + std::to_string(i) + ".";
      Wan wb;
      wb.mod = by[p + "mod"];
      wb.qkv = L(p + "sa.qkv"); wb.o = L(p + "sa.o");
      wb.qn = by[p + "sa.q_norm.w"]; wb.kn = by[p + "sa.k_norm.w"];
      wb.can_w = by[p + "ca.norm.w"]; wb.can_b = by[p + "ca.norm.b"];
      wb.cq = L(p + "ca.q"); wb.ckv = L(p + "ca.kv"); wb.co = L(p + "ca.o");
      wb.cqn = by[p + "ca.q_norm.w"]; wb.ckn = by[p + "ca.k_norm.w"];
      wb.ffn1 = L(p + "ffn1"); wb.ffn2 = L(p + "ffn2");
      m->wan.push_back(wb);
    }
    for (int i = 0; i < (cfg->model == FF_MODEL_MMDIT ? cfg->n_dual : 0); ++i)
      for (int k = 0; k < 2; ++k) {
        std::string p = "dual." + std::to_string(i) + (k == 0 ? ".img." : ".txt.");
        Stream st;
        st.mod = L(p + "mod"); st.qkv = L(p + "qkv"); st.o = L(p + "o");
        st.mlp1 = L(p + "mlp1"); st.mlp2 = L(p + "mlp2");
        st.qn = by[p + "q_norm.w"]; st.kn = by[p + "k_norm.w"];
        (k == 0 ? m->dual_img : m->dual_txt).push_back(st);
      }
    for (int j = 0; j < (cfg->model == FF_MODEL_MMDIT ? cfg->n_single : 0); ++j) {
      std::string p = "single." + std::to_string(j) + ".";
      Single sb;
      sb.mod = L(p + "mod"); sb.lin1 = L(p + "lin1"); sb.lin2 = L(p + "lin2");
      sb.qn = by[p + "q_norm.w"]; sb.kn = by[p + "k_norm.w"];
      m->single.push_back(sb);
    }
    *out = m.release();
    return FF_OK;
  });
}

int ff_dit_destroy(ff_dit* m) {
  delete m;
  return FF_OK;
}

static int check_forward_shape(const ff_dit* m, int64_t B, const int32_t grid[3], int64_t n_txt, int64_t n_prompts) {
  if (!m) return fail(FF_EINVAL, "ff_dit: null model");
  if (!grid) return fail(FF_EINVAL, "ff_dit: null grid");
  if (B < 1 || B > 65535) return fail(FF_EINVAL, "ff_dit: B=%lld outside [1, 65535]", (long long)B);
  if (grid[0] < 1 || grid[1] < 1 || grid[2] < 1) return fail(FF_EINVAL, "ff_dit: grid entries must be >= 1");
  if (n_txt < 1) return fail(FF_EINVAL, "ff_dit: n_txt must be >= 1");
  if (n_prompts < 1) return fail(FF_EINVAL, "ff_dit: n_prompts must be >= 1");
  if (grid[0] > kMaxAxis || grid[1] > kMaxAxis || grid[2] > kMaxAxis || n_txt > kMaxTxt || n_prompts > 65535)
    return fail(FF_EUNSUPPORTED, "ff_dit: grid axis, n_txt or n_prompts above its limit");
  const int64_t Ni = static_cast<int64_t>(grid[0]) * grid[1] * grid[2];
  if (Ni > kMaxRows || B * (Ni + n_txt) > kMaxRows || n_prompts * n_txt > kMaxRows)
    return fail(FF_EUNSUPPORTED, "ff_dit: more than %lld token rows in one forward", (long long)kMaxRows);
  if (m->cfg.dtype == FF_BF16 && (Ni % 8 || n_txt % 8))
    return fail(FF_EUNSUPPORTED, "ff_dit: bf16 token counts must be multiples of 8 (N_img=%lld, n_txt=%lld)", (long long)Ni, (long long)n_txt);
  return FF_OK;
}

int ff_dit_workspace_size(const ff_dit* m, int64_t B, const int32_t grid[3], int64_t n_txt, int64_t n_prompts,
                          size_t* bytes) {
  return guarded("ff_dit_workspace_size", [&]() -> int {
    FF_TRY(check_forward_shape(m, B, grid, n_txt, n_prompts));
    if (!bytes) return fail(FF_EINVAL, "ff_dit_workspace_size: null output");
    *bytes = plan(*m, B, grid, n_txt, n_prompts).total;
    return FF_OK;
  });
}

int ff_dit_forward(const ff_dit* m, const void* x, const void* txt, const int32_t* txt_index, int64_t n_prompts,
                   const void* cond, const float* t, const int32_t grid[3], int64_t B, int64_t n_txt, void* v_out,
                   void* txt_out, void* workspace, size_t ws_bytes, void* stream) {
  return guarded("ff_dit_forward", [&]() -> int {
    FF_TRY(check_forward_shape(m, B, grid, n_txt, n_prompts));
    const ff_dit_config& c = m->cfg;
    if (!x || !txt || !v_out) return fail(FF_EINVAL, "ff_dit_forward: null x, txt or v_out");
    if (!aligned16(x) || !aligned16(txt) || !aligned16(v_out) || (txt_out && !aligned16(txt_out)) ||
        (cond && !aligned16(cond)))
      return fail(FF_EINVAL, "ff_dit_forward: tensors must be 16-byte aligned");
    if (c.io_mode == FF_IO_LATENT) {
      if (!t) return fail(FF_EINVAL, "ff_dit_forward: latent mode needs t");
      if (txt_out) return fail(FF_EINVAL, "ff_dit_forward: txt_out must be NULL in latent mode");
      if (!txt_index && n_prompts != B) return fail(FF_EINVAL, "ff_dit_forward: txt_index NULL needs n_prompts == B");
      if (c.pooled_dim && !cond) return fail(FF_EINVAL, "ff_dit_forward: pooled_dim > 0 needs cond");
    } else {
      if (!cond) return fail(FF_EINVAL, "ff_dit_forward: hidden mode needs cond");
      if (txt_index || n_prompts != B) return fail(FF_EINVAL, "ff_dit_forward: hidden mode takes per-sample text (txt_index NULL, n_prompts == B)");
    }
    if (v_out == x || v_out == txt || (txt_out && (txt_out == x || txt_out == txt || txt_out == v_out)))
      return fail(FF_EINVAL, "ff_dit_forward: outputs may not alias inputs");
    Plan p = plan(*m, B, grid, n_txt, n_prompts);
    if (!workspace || ws_bytes < p.total)
      return fail(FF_EWORKSPACE, "ff_dit_forward: workspace of %zu bytes needed, %zu given", p.total, workspace ? ws_bytes : 0);
    if (!aligned16(workspace)) return fail(FF_EINVAL, "ff_dit_forward: workspace must be 16-byte aligned");
    if (c.model == FF_MODEL_WAN)
      return forward_wan(*m, p, x, txt, txt_index, t, grid, v_out, workspace, nullptr, static_cast<hipStream_t>(stream));
    return forward_mmdit(*m, p, x, txt, txt_index, cond, t, grid, v_out, txt_out, workspace, static_cast<hipStream_t>(stream));
  });
}

int ff_dit_context_size(const ff_dit* m, int64_t B, int64_t n_txt, size_t* bytes) {
  if (!m || !bytes) return fail(FF_EINVAL, "ff_dit_context_size: null model or output");
  if (m->cfg.model != FF_MODEL_WAN) return fail(FF_EUNSUPPORTED, "ff_dit_context_size: WAN models only");
  if (B < 1 || B > 65535 || n_txt < 1) return fail(FF_EINVAL, "ff_dit_context_size: bad B or n_txt");
  *bytes = static_cast<size_t>(2 * m->cfg.n_wan) * wan_kv_block_bytes(m->cfg, B, n_txt);
  return FF_OK;
}

int ff_dit_prepare_context(const ff_dit* m, const void* txt, const int32_t* txt_index, int64_t n_prompts,
                           const int32_t grid[3], int64_t B, int64_t n_txt, void* context, size_t context_bytes,
                           void* workspace, size_t ws_bytes, void* stream) {
  return guarded("ff_dit_prepare_context", [&]() -> int {
    FF_TRY(check_forward_shape(m, B, grid, n_txt, n_prompts));
    if (m->cfg.model != FF_MODEL_WAN) return fail(FF_EUNSUPPORTED, "ff_dit_prepare_context: WAN models only");
    if (!txt || !context) return fail(FF_EINVAL, "ff_dit_prepare_context: null txt or context");
    if (!aligned16(txt) || !aligned16(context)) return fail(FF_EINVAL, "ff_dit_prepare_context: txt and context must be 16-byte aligned");
    if (!txt_index && n_prompts != B) return fail(FF_EINVAL, "ff_dit_prepare_context: txt_index NULL needs n_prompts == B");
    const size_t kvb = wan_kv_block_bytes(m->cfg, B, n_txt);
    if (context_bytes < 2 * m->cfg.n_wan * kvb)
      return fail(FF_EWORKSPACE, "ff_dit_prepare_context: context of %zu bytes needed, %zu given", 2 * m->cfg.n_wan * kvb, context_bytes);
    Plan p = plan(*m, B, grid, n_txt, n_prompts);
    if (!workspace || ws_bytes < p.total)
      return fail(FF_EWORKSPACE, "ff_dit_prepare_context: workspace of %zu bytes needed, %zu given", p.total, workspace ? ws_bytes : 0);
    if (!aligned16(workspace)) return fail(FF_EINVAL, "ff_dit_prepare_context: workspace must be 16-byte aligned");
    const hipStream_t s = static_cast<hipStream_t>(stream);
    FF_TRY(wan_text_context(*m, p, txt, txt_index, workspace, s));
    char* store = static_cast<char*>(context);
    for (int i = 0; i < m->cfg.n_wan; ++i)
      FF_TRY(wan_cross_kv(*m, p, workspace, i, at(workspace, p.xtxt), store + 2 * i * kvb, store + (2 * i + 1) * kvb, s));
    return FF_OK;
  });
}

int ff_dit_forward_ctx(const ff_dit* m, const void* x, const void* context, size_t context_bytes, const float* t,
                       const int32_t grid[3], int64_t B, int64_t n_txt, void* v_out, void* workspace, size_t ws_bytes,
                       void* stream) {
  return guarded("ff_dit_forward_ctx", [&]() -> int {
    FF_TRY(check_forward_shape(m, B, grid, n_txt, 1));
    if (m->cfg.model != FF_MODEL_WAN) return fail(FF_EUNSUPPORTED, "ff_dit_forward_ctx: WAN models only");
    if (!x || !context || !t || !v_out) return fail(FF_EINVAL, "ff_dit_forward_ctx: null x, context, t or v_out");
    if (!aligned16(x) || !aligned16(context) || !aligned16(v_out))
      return fail(FF_EINVAL, "ff_dit_forward_ctx: tensors must be 16-byte aligned");
    if (v_out == x || v_out == context) return fail(FF_EINVAL, "ff_dit_forward_ctx: v_out may not alias an input");
    const size_t kvb = wan_kv_block_bytes(m->cfg, B, n_txt);
    if (context_bytes < 2 * m->cfg.n_wan * kvb)
      return fail(FF_EWORKSPACE, "ff_dit_forward_ctx: context of %zu bytes needed, %zu given", 2 * m->cfg.n_wan * kvb, context_bytes);
    Plan p = plan(*m, B, grid, n_txt, 1);   // the prompts' text buffers are not used here
    if (!workspace || ws_bytes < p.total)
      return fail(FF_EWORKSPACE, "ff_dit_forward_ctx: workspace of %zu bytes needed, %zu given", p.total, workspace ? ws_bytes : 0);
    if (!aligned16(workspace)) return fail(FF_EINVAL, "ff_dit_forward_ctx: workspace must be 16-byte aligned");
    return forward_wan(*m, p, x, nullptr, nullptr, t, grid, v_out, workspace, static_cast<const char*>(context),
                       static_cast<hipStream_t>(stream));
  });
}

}  // extern "C"
