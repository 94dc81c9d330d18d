// aj_varlen_block_fwd / aj_varlen_block_bwd, the checkpointed layer stack
// (aj_stack_fwd / aj_stack_bwd) and the embedding entry points.
//
// Forward:  a = RMSNorm(x) g1 -> qkv = a W_qkv^T -> RoPE(q, k) -> o = attention
//           -> x1 = x + o W_o^T -> b = RMSNorm(x1) g2 -> gu = b W_gu^T
//           -> s = silu(gate) * up -> y = x1 + s W_down^T
// Backward: the same chain reversed; weight gradients are GEMMs over the
// token axis accumulated into float32; the residual gradient stays float32.
#include <algorithm>
#include "ops.h"

namespace {

struct Saved {
  void *a, *qkv, *o, *x1, *b, *gu, *s;
  float *rstd1, *lse, *rstd2;
  size_t bytes;
};

Saved carve_saved(const aj_block_cfg &c, int n, void *base) {
  const size_t es = c.dtype == AJ_BF16 ? 2 : 4;
  const int64_t d = c.d_model, q = (int64_t)(c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  const int64_t hq = (int64_t)c.n_q_heads * c.head_dim, F = c.d_ff;
  aj::Carver cv(base);
  Saved s;
  s.a = cv.take<char>(n * d * es);
  s.qkv = cv.take<char>(n * q * es);
  s.o = cv.take<char>(n * hq * es);
  s.x1 = cv.take<char>(n * d * es);
  s.b = cv.take<char>(n * d * es);
  s.gu = cv.take<char>(n * 2 * F * es);
  s.s = cv.take<char>(n * F * es);
  s.rstd1 = cv.take<float>(n);
  s.lse = cv.take<float>((int64_t)c.n_q_heads * n);
  s.rstd2 = cv.take<float>(n);
  s.bytes = cv.bytes();
  return s;
}

struct BwdWs {
  void *dy_t, *ds, *dgu, *dx1_t, *dout, *dqkv;
  float *db, *dx1, *delta, *da, *dg_part, *splitk;
  size_t splitk_floats;
  size_t bytes;
};

BwdWs carve_bwd(const aj_block_cfg &c, int n, void *base) {
  const size_t es = c.dtype == AJ_BF16 ? 2 : 4;
  const int64_t d = c.d_model, q = (int64_t)(c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  const int64_t hq = (int64_t)c.n_q_heads * c.head_dim, F = c.d_ff;
  aj::Carver cv(base);
  BwdWs w;
  w.dy_t = cv.take<char>(n * d * es);
  w.ds = cv.take<char>(n * F * es);
  w.dgu = cv.take<char>(n * 2 * F * es);
  w.dx1_t = cv.take<char>(n * d * es);
  w.dout = cv.take<char>(n * hq * es);
  w.dqkv = cv.take<char>(n * q * es);
  w.db = cv.take<float>(n * d);
  w.dx1 = cv.take<float>(n * d);
  w.delta = cv.take<float>((int64_t)c.n_q_heads * n);
  w.da = cv.take<float>(n * d);
  w.dg_part = cv.take<float>(aj::rmsnorm_bwd_part_floats(n, (int)d));
  // split-K partials of the weight-gradient GEMMs (K = tokens)
  size_t sk = aj::gemm_split_floats((int)d, (int)F, n);
  sk = std::max(sk, aj::gemm_split_floats((int)(2 * F), (int)d, n));
  sk = std::max(sk, aj::gemm_split_floats((int)d, (int)hq, n));
  sk = std::max(sk, aj::gemm_split_floats((int)q, (int)d, n));
  w.splitk = cv.take<float>(sk > 0 ? sk : 1);
  w.splitk_floats = sk > 0 ? sk : 1;
  w.bytes = cv.bytes();
  return w;
}

// ---------------------------------------------------------------- LoRA
// Projection p in {0 qkv, 1 o, 2 gate_up, 3 down}: out = in W^T + u B^T with
// u = (in A^T)_s, (.)_s = scale * (.) rounded once to the storage type.  The
// rank-r term rides in the projection's own GEMM as a second reduction
// segment, so the output is written (and rounded) once; in the backward,
// d_in = d_out W + v A with v = (d_out B)_s likewise, and dB += d_out^T u,
// dA += v^T in are the adapters' gradients.
enum { kQkv = 0, kO = 1, kGu = 2, kDown = 3 };

struct LoraFwd {
  int r;
  float scale;
  const void *a[4], *b[4];
  void *u[4];         // [n, r] each: u of projection p, kept for the backward
  float *u32;         // [n, r] float32 product before the scale
};

struct LoraBwd {
  int r;
  float scale;
  const void *a[4], *b[4];
  const void *u[4];
  float *da[4], *db[4];
  float *v32;         // [n, r] d_out B
  void *vs;           // [n, r] v
  float *partial;     // split-K partials of dA / dB
  size_t partial_floats;
};

int proj_in(const aj_block_cfg &c, int p) {
  return p == kO ? c.n_q_heads * c.head_dim : p == kDown ? c.d_ff : c.d_model;
}
int proj_out(const aj_block_cfg &c, int p) {
  return p == kQkv ? (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim
                   : p == kGu ? 2 * c.d_ff : c.d_model;
}

// The adapters' part of the saved arena, placed after the block's own.
size_t carve_lora_saved(const aj_block_cfg &c, int r, int n, void *base, LoraFwd *lf) {
  const size_t es = c.dtype == AJ_BF16 ? 2 : 4;
  aj::Carver cv(base);
  for (int p = 0; p < 4; ++p) {
    void *u = cv.take<char>((int64_t)n * r * es);
    if (lf) lf->u[p] = u;
  }
  float *u32 = cv.take<float>((int64_t)n * r);
  if (lf) lf->u32 = u32;
  return cv.bytes();
}

// Split-K factor of the adapters' gradient GEMMs (a few output tiles, K =
// tokens): enough splits for ~2 workgroups per CU, at least 2048 k each.
int lora_split(int M, int N, int K) {
  const int tiles = ((M + 255) / 256) * ((N + 255) / 256);
  int S = (512 + tiles - 1) / tiles;
  S = std::min(S, std::min(K / 2048, 64));
  return S < 1 ? 1 : S;
}

size_t lora_split_floats(const aj_block_cfg &c, int r, int n) {
  size_t f = 0;
  for (int p = 0; p < 4; ++p) {
    const int o = proj_out(c, p), i = proj_in(c, p);
    const int sb = lora_split(o, r, n), sa = lora_split(r, i, n);
    if (sb > 1) f = std::max(f, (size_t)sb * o * r);   // dB
    if (sa > 1) f = std::max(f, (size_t)sa * r * i);   // dA
  }
  return f;
}

// The adapters' part of the backward workspace, placed after the block's own.
size_t carve_lora_bwd(const aj_block_cfg &c, int r, int n, void *base, LoraBwd *lb) {
  const size_t es = c.dtype == AJ_BF16 ? 2 : 4;
  aj::Carver cv(base);
  float *v32 = cv.take<float>((int64_t)n * r);
  void *vs = cv.take<char>((int64_t)n * r * es);
  const size_t sk = lora_split_floats(c, r, n);
  float *part = cv.take<float>(sk > 0 ? sk : 1);
  if (lb) { lb->v32 = v32; lb->vs = vs; lb->partial = part; lb->partial_floats = sk > 0 ? sk : 1; }
  return cv.bytes();
}

// u of projection p from its input (row stride k_in).
template <typename T>
int lora_u(const aj_block_cfg &c, const LoraFwd &lf, int p, const T *in, int n, hipStream_t st) {
  using namespace aj;
  const int k_in = proj_in(c, p), r = lf.r;
  Gemm g;
  g.M = n; g.N = r; g.K = k_in; g.A = in; g.lda = k_in; g.B = lf.a[p]; g.ldb = k_in;
  g.C = lf.u32; g.ldc = r; g.c_f32 = true;
  if (int rc = gemm<T>(g, st)) return rc;
  scale_cast<T>(lf.u32, (int64_t)n * r, lf.scale, (T *)lf.u[p], nullptr, st);
  return AJ_OK;
}

// The rank-r segment of the projection GEMM g (M = n, N = out): + u B^T.
void lora_fwd_seg(aj::Gemm &g, const LoraFwd *lf, int p) {
  if (!lf) return;
  g.A2 = lf->u[p]; g.lda2 = lf->r; g.B2 = lf->b[p]; g.ldb2 = lf->r; g.K2 = lf->r;
}

// From d_out of projection p (row stride n_out) and its input: dB += d_out^T u,
// v = (d_out B)_s, dA += v^T in.
template <typename T>
int lora_grads(const aj_block_cfg &c, const LoraBwd &lb, int p, const T *d_out, const T *in, int n,
               hipStream_t st) {
  using namespace aj;
  const int k_in = proj_in(c, p), n_out = proj_out(c, p), r = lb.r;
  int rc;
  Gemm g;   // dB [n_out, r] += d_out^T u
  g.M = n_out; g.N = r; g.K = n; g.A = d_out; g.lda = n_out; g.a_kmajor = false;
  g.B = lb.u[p]; g.ldb = r; g.b_kmajor = false; g.C = lb.db[p]; g.ldc = r;
  g.out = OUT_ACCUM_F32; g.split_k = lora_split(g.M, g.N, g.K); g.partial = lb.partial;
  g.partial_cap = lb.partial_floats;
  if ((rc = gemm<T>(g, st))) return rc;
  g = Gemm();   // v [n, r] = (d_out B)_s
  g.M = n; g.N = r; g.K = n_out; g.A = d_out; g.lda = n_out;
  g.B = lb.b[p]; g.ldb = r; g.b_kmajor = false; g.C = lb.v32; g.ldc = r; g.c_f32 = true;
  if ((rc = gemm<T>(g, st))) return rc;
  scale_cast<T>(lb.v32, (int64_t)n * r, lb.scale, (T *)lb.vs, nullptr, st);
  g = Gemm();   // dA [r, k_in] += v^T in
  g.M = r; g.N = k_in; g.K = n; g.A = lb.vs; g.lda = r; g.a_kmajor = false;
  g.B = in; g.ldb = k_in; g.b_kmajor = false; g.C = lb.da[p]; g.ldc = k_in;
  g.out = OUT_ACCUM_F32; g.split_k = lora_split(g.M, g.N, g.K); g.partial = lb.partial;
  g.partial_cap = lb.partial_floats;
  return gemm<T>(g, st);
}

// The rank-r segment of the input-gradient GEMM g (M = n, N = in): + v A.
void lora_bwd_seg(aj::Gemm &g, const LoraBwd *lb, int p, int k_in) {
  if (!lb) return;
  g.A2 = lb->vs; g.lda2 = lb->r; g.B2 = lb->a[p]; g.ldb2 = k_in; g.K2 = lb->r;
}

int check_cfg(const aj_block_cfg *c, const char *name) {
  AJ_REQUIRE(c, AJ_ERR_NULL, "%s: null cfg", name);
  AJ_REQUIRE(c->dtype == AJ_F32 || c->dtype == AJ_BF16, AJ_ERR_UNSUPPORTED, "%s: dtype %d", name,
             c->dtype);
  AJ_REQUIRE(c->d_model > 0 && c->d_model <= 8192 && c->d_model % 8 == 0, AJ_ERR_SHAPE,
             "%s: d_model %d (multiple of 8, at most 8192)", name, c->d_model);
  AJ_REQUIRE(c->n_q_heads > 0 && c->n_kv_heads > 0 && c->n_q_heads % c->n_kv_heads == 0,
             AJ_ERR_SHAPE, "%s: heads %d/%d", name, c->n_q_heads, c->n_kv_heads);
  AJ_REQUIRE(c->head_dim >= 8 && c->head_dim <= 128 && c->head_dim % 8 == 0, AJ_ERR_UNSUPPORTED,
             "%s: head_dim %d (8..128, multiple of 8)", name, c->head_dim);
  AJ_REQUIRE(c->d_ff > 0 && c->d_ff % 8 == 0, AJ_ERR_SHAPE, "%s: d_ff %d", name, c->d_ff);
  AJ_REQUIRE(c->rms_eps > 0 && c->rope_theta > 1, AJ_ERR_SHAPE, "%s: eps/theta", name);
  return AJ_OK;
}

int check_varlen(const aj_varlen *v, const char *name) {
  AJ_REQUIRE(v, AJ_ERR_NULL, "%s: null varlen", name);
  AJ_REQUIRE(v->n_tok >= 0 && v->n_seg >= 0 && (v->n_tok == 0 || v->n_seg > 0), AJ_ERR_SHAPE,
             "%s: n_tok %d n_seg %d", name, v->n_tok, v->n_seg);
  AJ_REQUIRE(v->n_tok == 0 || (v->cu_seqlens && v->pos), AJ_ERR_NULL, "%s: null offsets", name);
  return AJ_OK;
}

template <typename T>
int block_fwd(const aj_block_cfg &c, const aj_block_weights &w, const aj_varlen &v, const T *x,
              T *y, const Saved &sv, hipStream_t st, const LoraFwd *lf = nullptr) {
  using namespace aj;
  const int n = v.n_tok, d = c.d_model, hd = c.head_dim, Hq = c.n_q_heads, Hkv = c.n_kv_heads;
  const int qdim = (Hq + 2 * Hkv) * hd, F = c.d_ff;
  int r;
  // the projections read the transposed ([in][out]) weights when given
  const bool tw = sizeof(T) == 2 && !lf && w.w_qkv_t;
  auto weight = [&](Gemm &g, const void *w_kmajor, const void *w_t) {
    g.B = tw ? w_t : w_kmajor;
    g.ldb = tw ? g.N : g.K;
    g.b_kmajor = !tw;
  };
  rmsnorm_fwd<T>(x, (const T *)w.attn_norm, n, d, c.rms_eps, nullptr, 0, (T *)sv.a, sv.rstd1, st);
  Gemm g;
  g.M = n; g.N = qdim; g.K = d;
  g.A = sv.a; g.lda = d; weight(g, w.w_qkv, w.w_qkv_t); g.C = sv.qkv; g.ldc = qdim;
  if (lf && (r = lora_u<T>(c, *lf, kQkv, (const T *)sv.a, n, st))) return r;
  lora_fwd_seg(g, lf, kQkv);
  if ((r = gemm<T>(g, st))) return r;
  rope<T>((T *)sv.qkv, n, v.pos, Hq + Hkv, qdim, hd, c.rope_theta, false, st);
  AttnArgs at{n, v.n_seg, Hq, Hkv, hd, v.base, v.cu_seqlens, sv.qkv, sv.o, sv.lse,
              1.0f / sqrtf((float)hd)};
  if ((r = attn_fwd<T>(at, st))) return r;
  g = Gemm();
  g.M = n; g.N = d; g.K = Hq * hd;
  g.A = sv.o; g.lda = Hq * hd; weight(g, w.w_o, w.w_o_t); g.C = sv.x1; g.ldc = d; g.R = x;
  if (lf && (r = lora_u<T>(c, *lf, kO, (const T *)sv.o, n, st))) return r;
  lora_fwd_seg(g, lf, kO);
  if ((r = gemm<T>(g, st))) return r;
  rmsnorm_fwd<T>((const T *)sv.x1, (const T *)w.mlp_norm, n, d, c.rms_eps, nullptr, 0, (T *)sv.b,
                 sv.rstd2, st);
  g = Gemm();
  g.M = n; g.N = 2 * F; g.K = d;
  g.A = sv.b; g.lda = d; weight(g, w.w_gate_up, w.w_gate_up_t); g.C = sv.gu; g.ldc = 2 * F;
  if (lf && (r = lora_u<T>(c, *lf, kGu, (const T *)sv.b, n, st))) return r;
  lora_fwd_seg(g, lf, kGu);
  if ((r = gemm<T>(g, st))) return r;
  swiglu_fwd<T>((const T *)sv.gu, n, F, (T *)sv.s, st);
  g = Gemm();
  g.M = n; g.N = d; g.K = F;
  g.A = sv.s; g.lda = F; weight(g, w.w_down, w.w_down_t); g.C = y; g.ldc = d; g.R = sv.x1;
  if (lf && (r = lora_u<T>(c, *lf, kDown, (const T *)sv.s, n, st))) return r;
  lora_fwd_seg(g, lf, kDown);
  if ((r = gemm<T>(g, st))) return r;
  return check_launch("aj_varlen_block_fwd");
}

// With adapters (lb) the block's own weights and gains are frozen: no weight
// or gain gradients (gr is not read), the adapters' instead.
template <typename T>
int block_bwd(const aj_block_cfg &c, const aj_block_weights &w, const aj_varlen &v, const T *x,
              const Saved &sv, const float *dy, float *dx, const aj_block_grads &gr,
              const BwdWs &ws, hipStream_t st, const LoraBwd *lb = nullptr) {
  using namespace aj;
  const int n = v.n_tok, d = c.d_model, hd = c.head_dim, Hq = c.n_q_heads, Hkv = c.n_kv_heads;
  const int qdim = (Hq + 2 * Hkv) * hd, F = c.d_ff, hq = Hq * hd;
  const bool same = sizeof(T) == sizeof(float);
  int r;
  const T *dy_t = same ? (const T *)dy : (const T *)ws.dy_t;
  if (!same) cast_from_f32<T>(dy, (int64_t)n * d, (T *)ws.dy_t, st);
  const bool frozen = lb != nullptr;
  // MLP down projection
  Gemm g;
  if (!frozen) {
    g.M = d; g.N = F; g.K = n; g.A = dy_t; g.lda = d; g.a_kmajor = false;
    g.B = sv.s; g.ldb = F; g.b_kmajor = false; g.C = gr.w_down; g.ldc = F;
    g.out = OUT_ACCUM_F32; g.split_k = gemm_split_k(g.M, g.N, g.K); g.partial = ws.splitk;
    g.partial_cap = ws.splitk_floats;
    if ((r = gemm<T>(g, st))) return r;
  }
  if (lb && (r = lora_grads<T>(c, *lb, kDown, dy_t, (const T *)sv.s, n, st))) return r;
  g = Gemm();
  g.M = n; g.N = F; g.K = d; g.A = dy_t; g.lda = d;
  g.B = w.w_down; g.ldb = F; g.b_kmajor = false;
  lora_bwd_seg(g, lb, kDown, F);
  if constexpr (sizeof(T) == 2) {
    // d gate / d up straight from the float32 d s tile in the GEMM's epilogue
    g.C = ws.dgu; g.ldc = 2 * F; g.swiglu_gu = sv.gu;
    if ((r = gemm<T>(g, st))) return r;
  } else {
    g.C = ws.ds; g.ldc = F;
    if ((r = gemm<T>(g, st))) return r;
    swiglu_bwd<T, T>((const T *)ws.ds, (const T *)sv.gu, n, F, (T *)ws.dgu, st);
  }
  // gate/up projection
  if (!frozen) {
    g = Gemm();
    g.M = 2 * F; g.N = d; g.K = n; g.A = ws.dgu; g.lda = 2 * F; g.a_kmajor = false;
    g.B = sv.b; g.ldb = d; g.b_kmajor = false; g.C = gr.w_gate_up; g.ldc = d;
    g.out = OUT_ACCUM_F32; g.split_k = gemm_split_k(g.M, g.N, g.K); g.partial = ws.splitk;
    g.partial_cap = ws.splitk_floats;
    if ((r = gemm<T>(g, st))) return r;
  }
  if (lb && (r = lora_grads<T>(c, *lb, kGu, (const T *)ws.dgu, (const T *)sv.b, n, st))) return r;
  g = Gemm();
  g.M = n; g.N = d; g.K = 2 * F; g.A = ws.dgu; g.lda = 2 * F;
  g.B = w.w_gate_up; g.ldb = d; g.b_kmajor = false; g.C = ws.db; g.ldc = d; g.c_f32 = true;
  lora_bwd_seg(g, lb, kGu, d);
  if ((r = gemm<T>(g, st))) return r;
  rmsnorm_bwd<T>(ws.db, (const T *)sv.x1, sv.rstd2, (const T *)w.mlp_norm, n, d, nullptr, 0, 0, dy,
                 ws.dx1, same ? nullptr : (T *)ws.dx1_t, ws.dg_part,
                 frozen ? nullptr : gr.mlp_norm, st);
  const T *dx1_t = same ? (const T *)ws.dx1 : (const T *)ws.dx1_t;
  // attention output projection
  if (!frozen) {
    g = Gemm();
    g.M = d; g.N = hq; g.K = n; g.A = dx1_t; g.lda = d; g.a_kmajor = false;
    g.B = sv.o; g.ldb = hq; g.b_kmajor = false; g.C = gr.w_o; g.ldc = hq;
    g.out = OUT_ACCUM_F32; g.split_k = gemm_split_k(g.M, g.N, g.K); g.partial = ws.splitk;
    g.partial_cap = ws.splitk_floats;
    if ((r = gemm<T>(g, st))) return r;
  }
  if (lb && (r = lora_grads<T>(c, *lb, kO, dx1_t, (const T *)sv.o, n, st))) return r;
  g = Gemm();
  g.M = n; g.N = hq; g.K = d; g.A = dx1_t; g.lda = d;
  g.B = w.w_o; g.ldb = hq; g.b_kmajor = false; g.C = ws.dout; g.ldc = hq;
  lora_bwd_seg(g, lb, kO, hq);
  if ((r = gemm<T>(g, st))) return r;
  AttnBwdArgs ab{n, v.n_seg, Hq, Hkv, hd, v.base, v.cu_seqlens, sv.qkv, sv.o, ws.dout, sv.lse,
                 ws.delta, ws.dqkv, 1.0f / sqrtf((float)hd)};
  if ((r = attn_bwd<T>(ab, st))) return r;
  rope<T>((T *)ws.dqkv, n, v.pos, Hq + Hkv, qdim, hd, c.rope_theta, true, st);
  // qkv projection
  if (!frozen) {
    g = Gemm();
    g.M = qdim; g.N = d; g.K = n; g.A = ws.dqkv; g.lda = qdim; g.a_kmajor = false;
    g.B = sv.a; g.ldb = d; g.b_kmajor = false; g.C = gr.w_qkv; g.ldc = d;
    g.out = OUT_ACCUM_F32; g.split_k = gemm_split_k(g.M, g.N, g.K); g.partial = ws.splitk;
    g.partial_cap = ws.splitk_floats;
    if ((r = gemm<T>(g, st))) return r;
  }
  if (lb && (r = lora_grads<T>(c, *lb, kQkv, (const T *)ws.dqkv, (const T *)sv.a, n, st)))
    return r;
  g = Gemm();
  g.M = n; g.N = d; g.K = qdim; g.A = ws.dqkv; g.lda = qdim;
  g.B = w.w_qkv; g.ldb = d; g.b_kmajor = false; g.C = ws.da; g.ldc = d; g.c_f32 = true;
  lora_bwd_seg(g, lb, kQkv, d);
  if ((r = gemm<T>(g, st))) return r;
  rmsnorm_bwd<T>(ws.da, x, sv.rstd1, (const T *)w.attn_norm, n, d, nullptr, 0, 0, ws.dx1, dx,
                 nullptr, ws.dg_part, frozen ? nullptr : gr.attn_norm, st);
  return check_launch("aj_varlen_block_bwd");
}

int check_weights(const aj_block_weights *w, const char *name) {
  AJ_REQUIRE(w && w->attn_norm && w->w_qkv && w->w_o && w->mlp_norm && w->w_gate_up && w->w_down,
             AJ_ERR_NULL, "%s: null weight", name);
  const int nt = !!w->w_qkv_t + !!w->w_o_t + !!w->w_gate_up_t + !!w->w_down_t;
  AJ_REQUIRE(nt == 0 || nt == 4, AJ_ERR_NULL, "%s: %d of the 4 transposed weights given", name,
             nt);
  return AJ_OK;
}

int check_grads(const aj_block_grads *g, const char *name) {
  AJ_REQUIRE(g && g->attn_norm && g->w_qkv && g->w_o && g->mlp_norm && g->w_gate_up && g->w_down,
             AJ_ERR_NULL, "%s: null gradient", name);
  return AJ_OK;
}

LoraFwd lora_fwd_args(const aj_lora &lo, const LoraFwd &arena) {
  LoraFwd f = arena;
  f.r = lo.rank;
  f.scale = lo.scale;
  const void *a[4] = {lo.a_qkv, lo.a_o, lo.a_gate_up, lo.a_down};
  const void *b[4] = {lo.b_qkv, lo.b_o, lo.b_gate_up, lo.b_down};
  for (int p = 0; p < 4; ++p) { f.a[p] = a[p]; f.b[p] = b[p]; }
  return f;
}

LoraBwd lora_bwd_args(const aj_lora &lo, const aj_lora_grads &g, const LoraFwd &arena,
                      const LoraBwd &ws) {
  LoraBwd b = ws;
  const LoraFwd f = lora_fwd_args(lo, arena);
  b.r = f.r;
  b.scale = f.scale;
  float *da[4] = {g.a_qkv, g.a_o, g.a_gate_up, g.a_down};
  float *db[4] = {g.b_qkv, g.b_o, g.b_gate_up, g.b_down};
  for (int p = 0; p < 4; ++p) {
    b.a[p] = f.a[p]; b.b[p] = f.b[p]; b.u[p] = f.u[p]; b.da[p] = da[p]; b.db[p] = db[p];
  }
  return b;
}

// Layer l reads x (l == 0) or checkpoint slab l-1, and writes slab l (or y for
// the last layer): the checkpoints are the inputs of layers 1 .. n-1.
// lora (host array, or null): each layer's adapters; `la` their arena.
template <typename T>
int stack_fwd(const aj_block_cfg &c, int nl, const aj_block_weights *w, const aj_varlen &v,
              const T *x, T *y, T *ckpt, const Saved &sv, hipStream_t st,
              const aj_lora *lora = nullptr, const LoraFwd *la = nullptr) {
  const int64_t slab = (int64_t)v.n_tok * c.d_model;
  for (int l = 0; l < nl; ++l) {
    const T *in = l == 0 ? x : ckpt + (l - 1) * slab;
    T *out = l == nl - 1 ? y : ckpt + l * slab;
    LoraFwd lf;
    if (lora) lf = lora_fwd_args(lora[l], *la);
    if (int r = block_fwd<T>(c, w[l], v, in, out, sv, st, lora ? &lf : nullptr)) return r;
  }
  return AJ_OK;
}

// Last layer first, from the arena the forward left; every earlier layer is
// recomputed into the same arena right before its backward (its output slab
// is rewritten with the same values: the forward is deterministic).
template <typename T>
int stack_bwd(const aj_block_cfg &c, int nl, const aj_block_weights *w, const aj_varlen &v,
              const T *x, T *ckpt, const Saved &sv, const float *dy, float *dx,
              const aj_block_grads *g, const BwdWs &ws, hipStream_t st,
              const aj_lora *lora = nullptr, const aj_lora_grads *lg = nullptr,
              const LoraFwd *la = nullptr, const LoraBwd *lw = nullptr) {
  const int64_t slab = (int64_t)v.n_tok * c.d_model;
  static const aj_block_grads kNoGrads{};
  for (int l = nl - 1; l >= 0; --l) {
    const T *in = l == 0 ? x : ckpt + (l - 1) * slab;
    LoraFwd lf;
    LoraBwd lb;
    if (lora) {
      lf = lora_fwd_args(lora[l], *la);
      lb = lora_bwd_args(lora[l], lg[l], *la, *lw);
    }
    if (l < nl - 1)
      if (int r = block_fwd<T>(c, w[l], v, in, ckpt + l * slab, sv, st, lora ? &lf : nullptr))
        return r;
    if (int r = block_bwd<T>(c, w[l], v, in, sv, l == nl - 1 ? dy : dx, dx, g ? g[l] : kNoGrads,
                             ws, st, lora ? &lb : nullptr))
      return r;
  }
  return AJ_OK;
}

int check_lora(const aj_lora *lo, const aj_lora_grads *lg, int nl, const char *name) {
  AJ_REQUIRE(lo, AJ_ERR_NULL, "%s: null adapter array", name);
  for (int l = 0; l < nl; ++l) {
    const aj_lora &a = lo[l];
    AJ_REQUIRE(a.rank == lo[0].rank && a.scale == lo[0].scale, AJ_ERR_SHAPE,
               "%s: layer %d rank/scale differ from layer 0", name, l);
    AJ_REQUIRE(a.a_qkv && a.b_qkv && a.a_o && a.b_o && a.a_gate_up && a.b_gate_up && a.a_down &&
                   a.b_down,
               AJ_ERR_NULL, "%s: layer %d null adapter", name, l);
    if (lg)
      AJ_REQUIRE(lg[l].a_qkv && lg[l].b_qkv && lg[l].a_o && lg[l].b_o && lg[l].a_gate_up &&
                     lg[l].b_gate_up && lg[l].a_down && lg[l].b_down,
                 AJ_ERR_NULL, "%s: layer %d null adapter gradient", name, l);
  }
  AJ_REQUIRE(lo[0].rank >= 8 && lo[0].rank <= 256 && lo[0].rank % 8 == 0, AJ_ERR_SHAPE,
             "%s: rank %d (a multiple of 8 in 8..256)", name, lo[0].rank);
  return AJ_OK;
}

}  // namespace

extern "C" int aj_transpose_bf16(const void *src, int32_t rows, int32_t cols, void *dst,
                                 void *stream) {
  AJ_REQUIRE(src && dst, AJ_ERR_NULL, "aj_transpose_bf16: null pointer");
  AJ_REQUIRE(rows > 0 && cols > 0 && (int64_t)((rows + 63) / 64) * ((cols + 63) / 64) < (1ll << 31),
             AJ_ERR_SHAPE, "aj_transpose_bf16: %d x %d", rows, cols);
  aj::transpose16(src, rows, cols, dst, (hipStream_t)stream);
  return aj::check_launch("aj_transpose_bf16");
}

extern "C" size_t aj_block_saved_bytes(const aj_block_cfg *cfg, int32_t n_tok) {
  if (!cfg || n_tok < 0) return 0;
  return carve_saved(*cfg, n_tok, nullptr).bytes;
}

extern "C" size_t aj_block_workspace_bytes(const aj_block_cfg *cfg, int32_t n_tok, int32_t n_seg) {
  (void)n_seg;
  if (!cfg || n_tok < 0) return 0;
  return carve_bwd(*cfg, n_tok, nullptr).bytes;
}

extern "C" int aj_varlen_block_fwd(const aj_block_cfg *cfg, const aj_block_weights *w,
                                   const aj_varlen *vl, const void *x, void *y, void *saved,
                                   void *ws, size_t ws_bytes, void *stream) {
  const char *name = "aj_varlen_block_fwd";
  int r;
  if ((r = check_cfg(cfg, name)) || (r = check_varlen(vl, name)) || (r = check_weights(w, name)))
    return r;
  (void)ws; (void)ws_bytes;
  if (vl->n_tok == 0) return AJ_OK;
  AJ_REQUIRE(x && y && saved, AJ_ERR_NULL, "%s: null x/y/saved", name);
  Saved sv = carve_saved(*cfg, vl->n_tok, saved);
  hipStream_t st = (hipStream_t)stream;
  const aj::StageSpan span(st, AJ_KC_STAGE_BLOCK);
  if (cfg->dtype == AJ_BF16)
    return block_fwd<bf16_t>(*cfg, *w, *vl, (const bf16_t *)x, (bf16_t *)y, sv, st);
  return block_fwd<float>(*cfg, *w, *vl, (const float *)x, (float *)y, sv, st);
}

extern "C" int aj_varlen_block_bwd(const aj_block_cfg *cfg, const aj_block_weights *w,
                                   const aj_varlen *vl, const void *x, const void *saved,
                                   const float *dy, float *dx, const aj_block_grads *g, void *ws,
                                   size_t ws_bytes, void *stream) {
  const char *name = "aj_varlen_block_bwd";
  int r;
  if ((r = check_cfg(cfg, name)) || (r = check_varlen(vl, name)) || (r = check_weights(w, name)))
    return r;
  if ((r = check_grads(g, name))) return r;
  if (vl->n_tok == 0) return AJ_OK;
  AJ_REQUIRE(x && saved && dy && dx && ws, AJ_ERR_NULL, "%s: null x/saved/dy/dx/ws", name);
  BwdWs bw = carve_bwd(*cfg, vl->n_tok, ws);
  AJ_REQUIRE(ws_bytes >= bw.bytes, AJ_ERR_WORKSPACE, "%s: workspace %zu < %zu", name, ws_bytes,
             bw.bytes);
  Saved sv = carve_saved(*cfg, vl->n_tok, const_cast<void *>(saved));
  hipStream_t st = (hipStream_t)stream;
  const aj::StageSpan span(st, AJ_KC_STAGE_BLOCK);
  if (cfg->dtype == AJ_BF16)
    return block_bwd<bf16_t>(*cfg, *w, *vl, (const bf16_t *)x, sv, dy, dx, *g, bw, st);
  return block_bwd<float>(*cfg, *w, *vl, (const float *)x, sv, dy, dx, *g, bw, st);
}

extern "C" size_t aj_stack_ckpt_bytes(const aj_block_cfg *cfg, int32_t n_layers, int32_t n_tok) {
  if (!cfg || n_layers < 1 || n_tok < 0) return 0;
  const size_t es = cfg->dtype == AJ_BF16 ? 2 : 4;
  return (size_t)(n_layers - 1) * (size_t)n_tok * (size_t)cfg->d_model * es;
}

extern "C" int aj_stack_fwd(const aj_block_cfg *cfg, int32_t n_layers, const aj_block_weights *w,
                            const aj_varlen *vl, const void *x, void *y, void *ckpt, void *saved,
                            void *stream) {
  const char *name = "aj_stack_fwd";
  int r;
  if ((r = check_cfg(cfg, name)) || (r = check_varlen(vl, name))) return r;
  AJ_REQUIRE(n_layers >= 1 && n_layers <= 1024, AJ_ERR_SHAPE, "%s: n_layers %d", name, n_layers);
  AJ_REQUIRE(w, AJ_ERR_NULL, "%s: null weight array", name);
  for (int l = 0; l < n_layers; ++l)
    if ((r = check_weights(&w[l], name))) return r;
  if (vl->n_tok == 0) return AJ_OK;
  AJ_REQUIRE(x && y && saved && (ckpt || n_layers == 1), AJ_ERR_NULL,
             "%s: null x/y/ckpt/saved", name);
  Saved sv = carve_saved(*cfg, vl->n_tok, saved);
  hipStream_t st = (hipStream_t)stream;
  const aj::StageSpan span(st, AJ_KC_STAGE_BLOCK);
  if (cfg->dtype == AJ_BF16)
    return stack_fwd<bf16_t>(*cfg, n_layers, w, *vl, (const bf16_t *)x, (bf16_t *)y,
                             (bf16_t *)ckpt, sv, st);
  return stack_fwd<float>(*cfg, n_layers, w, *vl, (const float *)x, (float *)y, (float *)ckpt, sv,
                          st);
}

extern "C" int aj_stack_bwd(const aj_block_cfg *cfg, int32_t n_layers, const aj_block_weights *w,
                            const aj_varlen *vl, const void *x, void *ckpt, void *saved,
                            const float *dy, float *dx, const aj_block_grads *g, void *ws,
                            size_t ws_bytes, void *stream) {
  const char *name = "aj_stack_bwd";
  int r;
  if ((r = check_cfg(cfg, name)) || (r = check_varlen(vl, name))) return r;
  AJ_REQUIRE(n_layers >= 1 && n_layers <= 1024, AJ_ERR_SHAPE, "%s: n_layers %d", name, n_layers);
  AJ_REQUIRE(w && g, AJ_ERR_NULL, "%s: null weight or gradient array", name);
  for (int l = 0; l < n_layers; ++l)
    if ((r = check_weights(&w[l], name)) || (r = check_grads(&g[l], name))) return r;
  if (vl->n_tok == 0) return AJ_OK;
  AJ_REQUIRE(x && saved && dy && dx && ws && (ckpt || n_layers == 1), AJ_ERR_NULL,
             "%s: null x/ckpt/saved/dy/dx/ws", name);
  BwdWs bw = carve_bwd(*cfg, vl->n_tok, ws);
  AJ_REQUIRE(ws_bytes >= bw.bytes, AJ_ERR_WORKSPACE, "%s: workspace %zu < %zu", name, ws_bytes,
             bw.bytes);
  Saved sv = carve_saved(*cfg, vl->n_tok, saved);
  hipStream_t st = (hipStream_t)stream;
  const aj::StageSpan span(st, AJ_KC_STAGE_BLOCK);
  if (cfg->dtype == AJ_BF16)
    return stack_bwd<bf16_t>(*cfg, n_layers, w, *vl, (const bf16_t *)x, (bf16_t *)ckpt, sv, dy, dx,
                             g, bw, st);
  return stack_bwd<float>(*cfg, n_layers, w, *vl, (const float *)x, (float *)ckpt, sv, dy, dx, g,
                          bw, st);
}

extern "C" size_t aj_lora_saved_bytes(const aj_block_cfg *cfg, int32_t rank, int32_t n_tok) {
  if (!cfg || n_tok < 0 || rank < 1) return 0;
  return carve_saved(*cfg, n_tok, nullptr).bytes +
         carve_lora_saved(*cfg, rank, n_tok, nullptr, nullptr);
}

extern "C" size_t aj_lora_workspace_bytes(const aj_block_cfg *cfg, int32_t rank, int32_t n_tok) {
  if (!cfg || n_tok < 0 || rank < 1) return 0;
  return carve_bwd(*cfg, n_tok, nullptr).bytes +
         carve_lora_bwd(*cfg, rank, n_tok, nullptr, nullptr);
}

extern "C" int aj_stack_lora_fwd(const aj_block_cfg *cfg, int32_t n_layers,
                                 const aj_block_weights *w, const aj_lora *lora,
                                 const aj_varlen *vl, const void *x, void *y, void *ckpt,
                                 void *saved, void *stream) {
  const char *name = "aj_stack_lora_fwd";
  int r;
  if ((r = check_cfg(cfg, name)) || (r = check_varlen(vl, name))) return r;
  AJ_REQUIRE(n_layers >= 1 && n_layers <= 1024, AJ_ERR_SHAPE, "%s: n_layers %d", name, n_layers);
  AJ_REQUIRE(w, AJ_ERR_NULL, "%s: null weight array", name);
  for (int l = 0; l < n_layers; ++l)
    if ((r = check_weights(&w[l], name))) return r;
  if ((r = check_lora(lora, nullptr, n_layers, name))) return r;
  if (vl->n_tok == 0) return AJ_OK;
  AJ_REQUIRE(x && y && saved && (ckpt || n_layers == 1), AJ_ERR_NULL,
             "%s: null x/y/ckpt/saved", name);
  Saved sv = carve_saved(*cfg, vl->n_tok, saved);
  LoraFwd la{};
  carve_lora_saved(*cfg, lora[0].rank, vl->n_tok, (char *)saved + sv.bytes, &la);
  hipStream_t st = (hipStream_t)stream;
  const aj::StageSpan span(st, AJ_KC_STAGE_BLOCK);
  if (cfg->dtype == AJ_BF16)
    return stack_fwd<bf16_t>(*cfg, n_layers, w, *vl, (const bf16_t *)x, (bf16_t *)y,
                             (bf16_t *)ckpt, sv, st, lora, &la);
  return stack_fwd<float>(*cfg, n_layers, w, *vl, (const float *)x, (float *)y, (float *)ckpt, sv,
                          st, lora, &la);
}

extern "C" int aj_stack_lora_bwd(const aj_block_cfg *cfg, int32_t n_layers,
                                 const aj_block_weights *w, const aj_lora *lora,
                                 const aj_varlen *vl, const void *x, void *ckpt, void *saved,
                                 const float *dy, float *dx, const aj_lora_grads *g, void *ws,
                                 size_t ws_bytes, void *stream) {
  const char *name = "aj_stack_lora_bwd";
  int r;
  if ((r = check_cfg(cfg, name)) || (r = check_varlen(vl, name))) return r;
  AJ_REQUIRE(n_layers >= 1 && n_layers <= 1024, AJ_ERR_SHAPE, "%s: n_layers %d", name, n_layers);
  AJ_REQUIRE(w && g, AJ_ERR_NULL, "%s: null weight or gradient array", name);
  for (int l = 0; l < n_layers; ++l)
    if ((r = check_weights(&w[l], name))) return r;
  if ((r = check_lora(lora, g, n_layers, name))) return r;
  if (vl->n_tok == 0) return AJ_OK;
  AJ_REQUIRE(x && saved && dy && dx && ws && (ckpt || n_layers == 1), AJ_ERR_NULL,
             "%s: null x/ckpt/saved/dy/dx/ws", name);
  const int rank = lora[0].rank;
  BwdWs bw = carve_bwd(*cfg, vl->n_tok, ws);
  const size_t need = bw.bytes + carve_lora_bwd(*cfg, rank, vl->n_tok, nullptr, nullptr);
  AJ_REQUIRE(ws_bytes >= need, AJ_ERR_WORKSPACE, "%s: workspace %zu < %zu", name, ws_bytes, need);
  LoraBwd lw{};
  carve_lora_bwd(*cfg, rank, vl->n_tok, (char *)ws + bw.bytes, &lw);
  Saved sv = carve_saved(*cfg, vl->n_tok, saved);
  LoraFwd la{};
  carve_lora_saved(*cfg, rank, vl->n_tok, (char *)saved + sv.bytes, &la);
  hipStream_t st = (hipStream_t)stream;
  const aj::StageSpan span(st, AJ_KC_STAGE_BLOCK);
  if (cfg->dtype == AJ_BF16)
    return stack_bwd<bf16_t>(*cfg, n_layers, w, *vl, (const bf16_t *)x, (bf16_t *)ckpt, sv, dy, dx,
                             nullptr, bw, st, lora, g, &la, &lw);
  return stack_bwd<float>(*cfg, n_layers, w, *vl, (const float *)x, (float *)ckpt, sv, dy, dx,
                          nullptr, bw, st, lora, g, &la, &lw);
}
