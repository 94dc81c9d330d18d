// Around the actor update: GRPO advantages, the non-dummy episode filter
// (keeps the groups whose rewards are not all equal) and the AdamW step.
//
// Advantages: one workgroup per group, float32 block reductions (mean, then
// the sum of squared deviations), the keep decision by exact comparison.
// Selection: single-workgroup scans over episodes and timelines give every
// kept timeline its output slot and token base; one workgroup per output
// timeline then copies its tokens (coalesced) and writes the episode's
// advantage on its llm tokens (0 on the others, as in the input layout).  AdamW: one elementwise pass, 4 elements per thread
// where every stream is 16-byte aligned; HBM-bound (28 bytes per element, 30
// with a bfloat16 copy).
#include "ops.h"

namespace {

constexpr int kScan = 1024;

// Inclusive scan of one int per thread over the workgroup (blockDim.x == NT);
// *total receives the workgroup sum.
template <int NT>
AJ_DEV int scan_incl(int v, int *total) {
  __shared__ int part[NT / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) part[w] = x;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) {
    before += i < w ? part[i] : 0;
    all += part[i];
  }
  __syncthreads();
  *total = all;
  return x + before;
}

__global__ void zero_i32_kernel(int32_t *p) { *p = 0; }

template <int NT>
AJ_DEV float block_sum(float v, float *red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) s += red[i];
  return s;
}

__global__ __launch_bounds__(256) void grpo_kernel(int /*n_groups*/, const int32_t *off,
                                                   const float *reward, float eps, float *adv,
                                                   uint8_t *keep, int32_t *err) {
  __shared__ float red[4];
  __shared__ int diff;
  const int g = blockIdx.x;
  const int a = off[g], b = off[g + 1];
  if ((g == 0 && a != 0) || b < a) {
    if (threadIdx.x == 0 && err) atomicOr(err, AJ_DEVERR_OFFSETS);
    return;
  }
  const int n = b - a;
  if (threadIdx.x == 0) diff = 0;
  __syncthreads();
  const float r0 = n > 0 ? reward[a] : 0.f;
  float s = 0.f;
  for (int e = a + threadIdx.x; e < b; e += 256) {
    const float r = reward[e];
    s += r;
    if (r != r0) diff = 1;
  }
  s = block_sum<256>(s, red);
  const bool kept = n >= 2 && diff != 0;
  const float mu = n > 0 ? s / (float)n : 0.f;
  float q = 0.f;
  for (int e = a + threadIdx.x; e < b; e += 256) {
    const float d = reward[e] - mu;
    q += d * d;
  }
  q = block_sum<256>(q, red);
  const float sd = n >= 2 ? sqrtf(q / (float)(n - 1)) : 0.f;
  for (int e = a + threadIdx.x; e < b; e += 256) {
    adv[e] = kept ? (reward[e] - mu) / (sd + eps) : 0.f;
    keep[e] = kept ? 1 : 0;
  }
}

struct SelArgs {
  int n_traj, n_tl;
  int64_t n_tok;
  const int32_t *traj_tl_off;
  const int64_t *tl_tok_off;
  const int32_t *tok;
  const uint8_t *flags;
  const float *old_logprob;
  const uint8_t *keep;
  const float *ep_adv;
  aj_timelines_out out;
  int32_t *tl_traj;      // [n_tl] episode of each input timeline
  int32_t *tl_base;      // [n_traj] first output timeline of each kept episode
  int32_t *dst_src;      // [n_tl] input timeline of each output timeline
  int32_t *status;       // [1] 0 = offsets valid
  int32_t *err;
};

// offsets tile [0, n_tl) and [0, n_tok); every episode's timelines get its index
__global__ void sel_validate_kernel(SelArgs a) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  int bad = 0;
  if (t == 0)
    bad |= a.traj_tl_off[0] != 0 || a.traj_tl_off[a.n_traj] != a.n_tl ||
           a.tl_tok_off[0] != 0 || a.tl_tok_off[a.n_tl] != a.n_tok;
  if (t < a.n_traj) {
    const int lo = a.traj_tl_off[t], hi = a.traj_tl_off[t + 1];
    if (lo < 0 || lo > hi || hi > a.n_tl) {
      bad = 1;
    } else {
      for (int i = lo; i < hi; ++i) a.tl_traj[i] = t;
    }
  }
  if (t < a.n_tl && (a.tl_tok_off[t] < 0 || a.tl_tok_off[t] > a.tl_tok_off[t + 1] ||
                     a.tl_tok_off[t + 1] > a.n_tok))
    bad = 1;
  if (bad) {
    atomicOr(a.status, 1);
    if (a.err) atomicOr(a.err, AJ_DEVERR_OFFSETS);
  }
}

// episodes: output timeline offsets and each kept episode's first output timeline
__global__ __launch_bounds__(kScan) void sel_traj_kernel(SelArgs a) {
  const bool ok = *a.status == 0;
  int carry_e = 0, carry_t = 0;
  for (int c0 = 0; c0 < a.n_traj; c0 += kScan) {
    const int e = c0 + threadIdx.x;
    const int k = ok && e < a.n_traj && a.keep[e] ? 1 : 0;
    const int nt = k ? a.traj_tl_off[e + 1] - a.traj_tl_off[e] : 0;
    int te, tt;
    const int ie = scan_incl<kScan>(k, &te);
    const int it = scan_incl<kScan>(nt, &tt);
    if (k) {
      a.out.traj_tl_off[carry_e + ie - 1] = carry_t + it - nt;
      a.tl_base[e] = carry_t + it - nt;
    }
    carry_e += te;
    carry_t += tt;
  }
  if (threadIdx.x == 0) {
    a.out.traj_tl_off[carry_e] = carry_t;
    a.out.counts[0] = carry_e;
    a.out.counts[1] = carry_t;
  }
}

// timelines: output token offsets and the input timeline of every output slot
__global__ __launch_bounds__(kScan) void sel_tl_kernel(SelArgs a) {
  const bool ok = *a.status == 0;
  int64_t carry = 0;
  for (int c0 = 0; c0 < a.n_tl; c0 += kScan) {
    const int i = c0 + threadIdx.x;
    int len = 0, e = -1;
    if (ok && i < a.n_tl) {
      e = a.tl_traj[i];
      if (a.keep[e]) len = (int)(a.tl_tok_off[i + 1] - a.tl_tok_off[i]);
      else e = -1;
    }
    int tot;
    const int incl = scan_incl<kScan>(len, &tot);
    if (e >= 0) {
      const int dst = a.tl_base[e] + (i - a.traj_tl_off[e]);
      a.out.tl_tok_off[dst] = carry + incl - len;
      a.dst_src[dst] = i;
    }
    carry += tot;
  }
  if (threadIdx.x == 0) {
    const int n_out = ok ? (int)a.out.counts[1] : 0;
    a.out.tl_tok_off[n_out] = carry;
    a.out.counts[2] = carry;
    if (!ok) {
      a.out.counts[0] = a.out.counts[1] = 0;
      a.out.traj_tl_off[0] = 0;
    }
  }
}

__global__ __launch_bounds__(256) void sel_copy_kernel(SelArgs a) {
  const int dst = blockIdx.x;
  if (*a.status != 0 || dst >= a.out.counts[1]) return;
  const int src = a.dst_src[dst];
  const int64_t s0 = a.tl_tok_off[src], n = a.tl_tok_off[src + 1] - s0;
  const int64_t d0 = a.out.tl_tok_off[dst];
  const float adv = a.ep_adv[a.tl_traj[src]];
  for (int64_t j = threadIdx.x; j < n; j += 256) {
    a.out.tok[d0 + j] = a.tok[s0 + j];
    a.out.flags[d0 + j] = a.flags[s0 + j];
    a.out.old_logprob[d0 + j] = a.old_logprob[s0 + j];
    a.out.adv[d0 + j] = (a.flags[s0 + j] & 3) == AJ_AUTHOR_LLM ? adv : 0.f;
  }
}

struct SelWs {
  int32_t *tl_traj, *tl_base, *dst_src, *status;
  size_t bytes;
};

SelWs carve_sel(int n_traj, int n_tl, void *base) {
  aj::Carver cv(base);
  SelWs w;
  w.tl_traj = cv.take<int32_t>(n_tl > 0 ? n_tl : 1);
  w.tl_base = cv.take<int32_t>(n_traj > 0 ? n_traj : 1);
  w.dst_src = cv.take<int32_t>(n_tl > 0 ? n_tl : 1);
  w.status = cv.take<int32_t>(1);
  w.bytes = cv.bytes();
  return w;
}

template <typename TC, bool VEC>
__global__ __launch_bounds__(256) void adamw_kernel(int64_t n, float *p, const float *g, float *m,
                                                    float *v, float lr, float b1, float b2,
                                                    float eps, float wd, float c1, float c2,
                                                    float gs, TC *copy) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  auto one = [&](float &pp, float gg, float &mm, float &vv) {
    gg *= gs;
    mm = b1 * mm + (1.f - b1) * gg;
    vv = b2 * vv + (1.f - b2) * gg * gg;
    pp = pp - lr * wd * pp - lr * (mm / c1) / (sqrtf(vv / c2) + eps);
  };
  if (VEC) {
    const int64_t n4 = n / 4;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
      float4 pp = reinterpret_cast<float4 *>(p)[i];
      const float4 gg = reinterpret_cast<const float4 *>(g)[i];
      float4 mm = reinterpret_cast<float4 *>(m)[i], vv = reinterpret_cast<float4 *>(v)[i];
      one(pp.x, gg.x, mm.x, vv.x);
      one(pp.y, gg.y, mm.y, vv.y);
      one(pp.z, gg.z, mm.z, vv.z);
      one(pp.w, gg.w, mm.w, vv.w);
      reinterpret_cast<float4 *>(p)[i] = pp;
      reinterpret_cast<float4 *>(m)[i] = mm;
      reinterpret_cast<float4 *>(v)[i] = vv;
      if (copy) {
        stf(copy + 4 * i, pp.x); stf(copy + 4 * i + 1, pp.y);
        stf(copy + 4 * i + 2, pp.z); stf(copy + 4 * i + 3, pp.w);
      }
    }
    for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
      one(p[i], g[i], m[i], v[i]);
      if (copy) stf(copy + i, p[i]);
    }
  } else {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
      one(p[i], g[i], m[i], v[i]);
      if (copy) stf(copy + i, p[i]);
    }
  }
}

bool al16(const void *p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

extern "C" int aj_grpo_advantages(int32_t n_groups, const int32_t *group_off, const float *reward,
                                  float eps, float *ep_adv, uint8_t *ep_keep, int32_t *err,
                                  void *stream) {
  const char *name = "aj_grpo_advantages";
  AJ_REQUIRE(n_groups >= 0, AJ_ERR_SHAPE, "%s: n_groups %d", name, n_groups);
  if (n_groups == 0) return AJ_OK;
  AJ_REQUIRE(group_off && reward && ep_adv && ep_keep, AJ_ERR_NULL, "%s: null pointer", name);
  AJ_REQUIRE(eps >= 0.f, AJ_ERR_SHAPE, "%s: eps %g", name, eps);
  hipStream_t st = (hipStream_t)stream;
  const int tk = aj::timing_begin(st, AJ_KC_SELECT, 0.0);
  grpo_kernel<<<n_groups, 256, 0, st>>>(n_groups, group_off, reward, eps, ep_adv, ep_keep, err);
  aj::timing_end(st, tk);
  return aj::check_launch(name);
}

extern "C" size_t aj_select_workspace_bytes(int32_t n_traj, int32_t n_tl) {
  if (n_traj < 0 || n_tl < 0) return 0;
  return carve_sel(n_traj, n_tl, nullptr).bytes;
}

extern "C" int aj_select_episodes(const aj_timelines *in, const uint8_t *keep, const float *ep_adv,
                                  aj_timelines_out *out, int32_t *err, void *ws, size_t ws_bytes,
                                  void *stream) {
  const char *name = "aj_select_episodes";
  AJ_REQUIRE(in && out, AJ_ERR_NULL, "%s: null argument struct", name);
  AJ_REQUIRE(in->n_traj >= 0 && in->n_tl >= 0 && in->n_tok >= 0 && in->n_tok < (int64_t)1 << 31,
             AJ_ERR_SHAPE, "%s: sizes", name);
  AJ_REQUIRE(in->n_tl == 0 || in->n_traj > 0, AJ_ERR_SHAPE, "%s: timelines without episodes", name);
  AJ_REQUIRE(in->traj_tl_off && in->tl_tok_off && out->traj_tl_off && out->tl_tok_off &&
                 out->counts,
             AJ_ERR_NULL, "%s: null offsets", name);
  AJ_REQUIRE(in->n_traj == 0 || (keep && ep_adv), AJ_ERR_NULL, "%s: null keep / ep_adv", name);
  AJ_REQUIRE(in->n_tok == 0 || (in->tok && in->flags && in->old_logprob && out->tok &&
                                out->flags && out->old_logprob && out->adv),
             AJ_ERR_NULL, "%s: null token arrays", name);
  SelWs w = carve_sel(in->n_traj, in->n_tl, ws);
  AJ_REQUIRE(ws && ws_bytes >= w.bytes, AJ_ERR_WORKSPACE, "%s: workspace %zu < %zu", name,
             ws_bytes, w.bytes);
  hipStream_t st = (hipStream_t)stream;
  SelArgs a{in->n_traj, in->n_tl, in->n_tok, in->traj_tl_off, in->tl_tok_off, in->tok,
            in->flags, in->old_logprob, keep, ep_adv, *out, w.tl_traj, w.tl_base, w.dst_src,
            w.status, err};
  const int tk = aj::timing_begin(st, AJ_KC_SELECT, 0.0);
  zero_i32_kernel<<<1, 1, 0, st>>>(w.status);
  const int nv = (in->n_traj > in->n_tl ? in->n_traj : in->n_tl) + 1;
  sel_validate_kernel<<<(nv + 255) / 256, 256, 0, st>>>(a);
  sel_traj_kernel<<<1, kScan, 0, st>>>(a);
  sel_tl_kernel<<<1, kScan, 0, st>>>(a);
  if (in->n_tl > 0) sel_copy_kernel<<<in->n_tl, 256, 0, st>>>(a);
  aj::timing_end(st, tk);
  return aj::check_launch(name);
}

extern "C" int aj_adamw_step(int64_t n, float *param, const float *grad, float *m, float *v,
                             float lr, float beta1, float beta2, float eps, float weight_decay,
                             int32_t step, float grad_scale, void *param_copy, int copy_dtype,
                             void *stream) {
  const char *name = "aj_adamw_step";
  AJ_REQUIRE(n >= 0, AJ_ERR_SHAPE, "%s: n %lld", name, (long long)n);
  if (n == 0) return AJ_OK;
  AJ_REQUIRE(param && grad && m && v, AJ_ERR_NULL, "%s: null pointer", name);
  AJ_REQUIRE(step >= 1, AJ_ERR_SHAPE, "%s: step %d (counts from 1)", name, step);
  AJ_REQUIRE(beta1 >= 0.f && beta1 < 1.f && beta2 >= 0.f && beta2 < 1.f && eps >= 0.f,
             AJ_ERR_SHAPE, "%s: betas / eps", name);
  AJ_REQUIRE(!param_copy || copy_dtype == AJ_F32 || copy_dtype == AJ_BF16, AJ_ERR_UNSUPPORTED,
             "%s: copy dtype %d", name, copy_dtype);
  hipStream_t st = (hipStream_t)stream;
  const float c1 = 1.f - powf(beta1, (float)step), c2 = 1.f - powf(beta2, (float)step);
  const bool vec = al16(param) && al16(grad) && al16(m) && al16(v) &&
                   (!param_copy || ((uintptr_t)param_copy & 7) == 0);
  const int64_t work = vec ? (n + 3) / 4 : n;
  const unsigned grid = (unsigned)(work < 256 * 4096 ? (work + 255) / 256 : 4096);
  const int tk = aj::timing_begin(st, AJ_KC_ADAMW, 0.0);
  if (copy_dtype == AJ_BF16) {
    bf16_t *c = (bf16_t *)param_copy;
    if (vec) adamw_kernel<bf16_t, true><<<grid, 256, 0, st>>>(n, param, grad, m, v, lr, beta1, beta2, eps, weight_decay, c1, c2, grad_scale, c);
    else adamw_kernel<bf16_t, false><<<grid, 256, 0, st>>>(n, param, grad, m, v, lr, beta1, beta2, eps, weight_decay, c1, c2, grad_scale, c);
  } else {
    float *c = (float *)param_copy;
    if (vec) adamw_kernel<float, true><<<grid, 256, 0, st>>>(n, param, grad, m, v, lr, beta1, beta2, eps, weight_decay, c1, c2, grad_scale, c);
    else adamw_kernel<float, false><<<grid, 256, 0, st>>>(n, param, grad, m, v, lr, beta1, beta2, eps, weight_decay, c1, c2, grad_scale, c);
  }
  aj::timing_end(st, tk);
  return aj::check_launch(name);
}
