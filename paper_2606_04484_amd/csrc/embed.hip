// Embedding gather x = E[tok] and its backward, the scatter-add
// dE[v] += sum over positions p with tok[p] == v of dx[p], made
// deterministic without float atomics:
//   1. keys (token << 32 | position) are sorted ascending by a bitonic
//      network (LDS-resident 4096-key chunks, global passes for the longer
//      strides).  The keys are unique, so the sorted order -- runs of equal
//      token, positions ascending inside a run -- does not depend on how the
//      sort is scheduled;
//   2. the sorted rows are cut into tiles of 256; one wave per (tile,
//      256-column slice) walks its rows in order and sums each run of equal
//      token.  A run that begins and ends inside the tile is added to dE
//      right there (it has no other owner); the piece of a run that crosses
//      into the next tile goes to a tile slot: slot 1 the piece of a run
//      that begins in the tile, slot 0 the piece of one that began earlier
//      (the whole tile when the run spans it);
//   3. a run that crosses tile boundaries is finished by the boundary it
//      crosses first: slot 1 of its first tile, then slot 0 of each later
//      tile in order, added to dE once.
// Each dE row is therefore written by one owner, with the same sum order on
// every call.
#include "ops.h"

namespace aj {
namespace {

constexpr int kChunk = 4096;           // keys per LDS-resident bitonic chunk (32 KB)
constexpr int kSortThreads = 512;
constexpr int kTile = 256;             // sorted rows per reduction tile
constexpr int kWaveCols = 256;         // columns per wave: 64 lanes x 4
constexpr int kTileWaves = 4;
constexpr uint32_t kNoTok = 0xffffffffu;

AJ_DEV uint32_t key_tok(uint64_t k) { return (uint32_t)(k >> 32); }
AJ_DEV uint32_t key_pos(uint64_t k) { return (uint32_t)k; }

template <typename T>
__global__ __launch_bounds__(256) void embed_fwd_kernel(const int32_t *tok, int n, const T *emb,
                                                        int d, int vocab, T *x, int32_t *err) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= n) return;
  const int t = tok[row];
  const bool ok = t >= 0 && t < vocab;
  if (!ok && lane == 0 && err) atomicOr(err, AJ_DEVERR_TOKEN_RANGE);
  const T *src = emb + (int64_t)(ok ? t : 0) * d;
  T *dst = x + (int64_t)row * d;
  for (int c = lane; c < d; c += 64) dst[c] = ok ? src[c] : T(0);
}

// keys[i] = tok << 32 | i for i < n (token field kNoTok when out of range:
// those rows sort to the end and are skipped); padding up to n2 = all ones.
__global__ __launch_bounds__(256) void embed_keys_kernel(const int32_t *tok, int n, int n2,
                                                         int vocab, uint64_t *keys) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n2; i += gridDim.x * 256) {
    uint64_t k = ~0ull;
    if (i < n) {
      const int t = tok[i];
      const uint32_t tt = (t >= 0 && t < vocab) ? (uint32_t)t : kNoTok;
      k = ((uint64_t)tt << 32) | (uint32_t)i;
    }
    keys[i] = k;
  }
}

// One compare-exchange step (stage k, stride j) over the chunk in LDS; pair
// q joins i = (q / j) * 2j + q % j with i + j, ascending where bit k of the
// global index of i is clear.
AJ_DEV void bitonic_step(uint64_t *s, int64_t base, int k, int j) {
  const int lj = __ffs(j) - 1;
  for (int q = threadIdx.x; q < kChunk / 2; q += kSortThreads) {
    const int i = ((q >> lj) << (lj + 1)) | (q & (j - 1));
    const bool asc = ((base + i) & k) == 0;
    const uint64_t a = s[i], b = s[i + j];
    if ((a > b) == asc) {
      s[i] = b;
      s[i + j] = a;
    }
  }
  __syncthreads();
}

// k_fixed == 0: every stage k <= kChunk of the network on each chunk;
// else the strides j < kChunk of stage k_fixed (> kChunk).
__global__ __launch_bounds__(kSortThreads) void bitonic_chunk_kernel(uint64_t *keys, int k_fixed) {
  __shared__ uint64_t s[kChunk];
  const int64_t base = (int64_t)blockIdx.x * kChunk;
  for (int t = threadIdx.x; t < kChunk; t += kSortThreads) s[t] = keys[base + t];
  __syncthreads();
  if (k_fixed == 0) {
    for (int k = 2; k <= kChunk; k <<= 1)
      for (int j = k >> 1; j > 0; j >>= 1) bitonic_step(s, base, k, j);
  } else {
    for (int j = kChunk >> 1; j > 0; j >>= 1) bitonic_step(s, base, k_fixed, j);
  }
  for (int t = threadIdx.x; t < kChunk; t += kSortThreads) keys[base + t] = s[t];
}

// One global compare-exchange step (stride j >= kChunk) of stage k.
__global__ __launch_bounds__(256) void bitonic_global_kernel(uint64_t *keys, int half, int k,
                                                             int j) {
  const int q = blockIdx.x * 256 + threadIdx.x;
  if (q >= half) return;
  const int lj = __ffs(j) - 1;
  const int i = ((q >> lj) << (lj + 1)) | (q & (j - 1));
  const bool asc = (i & k) == 0;
  const uint64_t a = keys[i], b = keys[i + j];
  if ((a > b) == asc) {
    keys[i] = b;
    keys[i + j] = a;
  }
}

AJ_DEV void add4(float4 &a, const float4 &b) {
  a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
}

// Step 2: one wave per (tile, 256-column slice); lane l owns columns
// col0 .. col0+3.  piece: [n_tiles][2][d].
__global__ __launch_bounds__(256) void embed_tile_kernel(const uint64_t *keys, int n,
                                                         const float *dx, int d, float *demb,
                                                         float *piece) {
  __shared__ uint64_t sk[kTile];
  const int tile = blockIdx.x;
  const int r0 = tile * kTile, r1 = min(n, r0 + kTile);
  for (int t = threadIdx.x; t < r1 - r0; t += 256) sk[t] = keys[r0 + t];
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col0 = (blockIdx.y * kTileWaves + wave) * kWaveCols + 4 * lane;
  if (col0 >= d) return;
  const uint32_t prev_tok = r0 > 0 ? key_tok(keys[r0 - 1]) : kNoTok;
  const uint32_t next_tok = r1 < n ? key_tok(keys[r1]) : kNoTok;
  float *slot0 = piece + ((int64_t)tile * 2) * d + col0;
  float *slot1 = slot0 + d;
  uint32_t cur = key_tok(sk[0]);
  bool began_before = cur == prev_tok;         // the first run started in an earlier tile
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  auto flush = [&](bool continues) {
    if (cur == kNoTok) return;
    if (began_before) {
      *(float4 *)slot0 = acc;                    // head piece (or the whole tile)
    } else if (continues) {
      *(float4 *)slot1 = acc;                    // tail piece of a run that begins here
    } else {
      float4 *o = (float4 *)(demb + (int64_t)cur * d + col0);
      float4 v = *o;
      add4(v, acc);
      *o = v;
    }
  };
  for (int r = r0; r < r1; r += 8) {
    float4 v[8];
    uint32_t tt[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int rr = r + u;
      const uint64_t k = rr < r1 ? sk[rr - r0] : ~0ull;
      tt[u] = key_tok(k);
      v[u] = (rr < r1 && tt[u] != kNoTok)
                 ? *(const float4 *)(dx + (int64_t)key_pos(k) * d + col0)
                 : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (r + u >= r1) break;
      if (tt[u] != cur) {
        flush(false);
        cur = tt[u];
        began_before = false;
        acc = make_float4(0.f, 0.f, 0.f, 0.f);
      }
      add4(acc, v[u]);
    }
  }
  flush(cur == next_tok);
}

// Step 3: the run crossing boundary b = (blockIdx.x + 1) * kTile, if it
// crosses no earlier boundary; one thread per 4 columns.
__global__ __launch_bounds__(256) void embed_cross_kernel(const uint64_t *keys, int n, int n_tiles,
                                                          int d, const float *piece, float *demb) {
  const int bt = blockIdx.x + 1;
  const int64_t b = (int64_t)bt * kTile;
  if (b >= n) return;
  const uint32_t t = key_tok(keys[b - 1]);
  if (t == kNoTok || key_tok(keys[b]) != t) return;
  if (bt > 1 && key_tok(keys[b - kTile - 1]) == t) return;     // crosses b - kTile too
  const int col0 = (blockIdx.y * 256 + threadIdx.x) * 4;
  if (col0 >= d) return;
  float4 acc = *(const float4 *)(piece + ((int64_t)(bt - 1) * 2 + 1) * d + col0);
  for (int u = bt;; ++u) {
    add4(acc, *(const float4 *)(piece + ((int64_t)u * 2) * d + col0));
    const int64_t e = (int64_t)(u + 1) * kTile;
    if (u + 1 >= n_tiles || e >= n || key_tok(keys[e]) != t) break;
  }
  float4 *o = (float4 *)(demb + (int64_t)t * d + col0);
  float4 v = *o;
  add4(v, acc);
  *o = v;
}

int64_t sort_len(int n) {
  int64_t n2 = kChunk;
  while (n2 < n) n2 <<= 1;
  return n2;
}

struct EmbedWs {
  uint64_t *keys;
  float *piece;
  size_t bytes;
};

EmbedWs carve_embed(void *ws, int n, int d) {
  Carver c(ws);
  EmbedWs w;
  w.keys = c.take<uint64_t>(sort_len(n));
  const int64_t tiles = (n + kTile - 1) / kTile;
  w.piece = c.take<float>(2 * tiles * (int64_t)d);
  w.bytes = c.bytes();
  return w;
}

}  // namespace

template <typename T>
void embed_fwd(const int32_t *tok, int n, const T *emb, int d, int vocab, T *x, int32_t *err,
               hipStream_t s) {
  if (n > 0) embed_fwd_kernel<T><<<(n + 3) / 4, 256, 0, s>>>(tok, n, emb, d, vocab, x, err);
}
template void embed_fwd<float>(const int32_t *, int, const float *, int, int, float *, int32_t *,
                               hipStream_t);
template void embed_fwd<bf16_t>(const int32_t *, int, const bf16_t *, int, int, bf16_t *,
                                int32_t *, hipStream_t);

}  // namespace aj

extern "C" int aj_embed_fwd(const int32_t *tok, int32_t n_tok, const void *emb, int32_t d,
                            int32_t vocab, int dtype, void *x, int32_t *err, void *stream) {
  AJ_REQUIRE(n_tok >= 0 && d > 0 && vocab > 0, AJ_ERR_SHAPE, "aj_embed_fwd: sizes");
  if (n_tok == 0) return AJ_OK;
  AJ_REQUIRE(tok && emb && x, AJ_ERR_NULL, "aj_embed_fwd: null pointer");
  hipStream_t st = (hipStream_t)stream;
  if (dtype == AJ_BF16)
    aj::embed_fwd<bf16_t>(tok, n_tok, (const bf16_t *)emb, d, vocab, (bf16_t *)x, err, st);
  else if (dtype == AJ_F32)
    aj::embed_fwd<float>(tok, n_tok, (const float *)emb, d, vocab, (float *)x, err, st);
  else
    return aj::fail(AJ_ERR_UNSUPPORTED, "aj_embed_fwd: dtype %d", dtype);
  return aj::check_launch("aj_embed_fwd");
}

extern "C" size_t aj_embed_bwd_workspace_bytes(int32_t n_tok, int32_t d) {
  if (n_tok < 0 || d <= 0) return 0;
  return aj::carve_embed(nullptr, n_tok, d).bytes;
}

extern "C" int aj_embed_bwd(const int32_t *tok, int32_t n_tok, const float *dx, int32_t d,
                            int32_t vocab, float *d_emb, void *ws, size_t ws_bytes,
                            void *stream) {
  using namespace aj;
  AJ_REQUIRE(n_tok >= 0 && d > 0 && vocab > 0, AJ_ERR_SHAPE, "aj_embed_bwd: sizes");
  AJ_REQUIRE(n_tok <= (1 << 30), AJ_ERR_UNSUPPORTED, "aj_embed_bwd: n_tok %d > 2^30", n_tok);
  AJ_REQUIRE(d % 4 == 0, AJ_ERR_UNSUPPORTED, "aj_embed_bwd: d %d not a multiple of 4", d);
  if (n_tok == 0) return AJ_OK;
  AJ_REQUIRE(tok && dx && d_emb && ws, AJ_ERR_NULL, "aj_embed_bwd: null pointer");
  AJ_REQUIRE(((uintptr_t)dx & 15) == 0 && ((uintptr_t)d_emb & 15) == 0, AJ_ERR_UNSUPPORTED,
             "aj_embed_bwd: dx and d_emb must be 16-byte aligned");
  const EmbedWs w = carve_embed(ws, n_tok, d);
  AJ_REQUIRE(ws_bytes >= w.bytes, AJ_ERR_WORKSPACE, "aj_embed_bwd: workspace %zu < %zu",
             ws_bytes, w.bytes);
  hipStream_t s = (hipStream_t)stream;
  const int64_t n2 = sort_len(n_tok);
  embed_keys_kernel<<<(int)std::min<int64_t>((n2 + 255) / 256, 4096), 256, 0, s>>>(
      tok, n_tok, (int)n2, vocab, w.keys);
  const int chunks = (int)(n2 / kChunk);
  bitonic_chunk_kernel<<<chunks, kSortThreads, 0, s>>>(w.keys, 0);
  for (int64_t k = 2 * kChunk; k <= n2; k <<= 1) {
    for (int64_t j = k >> 1; j >= kChunk; j >>= 1)
      bitonic_global_kernel<<<(int)((n2 / 2 + 255) / 256), 256, 0, s>>>(w.keys, (int)(n2 / 2),
                                                                          (int)k, (int)j);
    bitonic_chunk_kernel<<<chunks, kSortThreads, 0, s>>>(w.keys, (int)k);
  }
  const int tiles = (n_tok + kTile - 1) / kTile;
  const int col_blocks = (d + kTileWaves * kWaveCols - 1) / (kTileWaves * kWaveCols);
  embed_tile_kernel<<<dim3(tiles, col_blocks), 256, 0, s>>>(w.keys, n_tok, dx, d, d_emb, w.piece);
  if (tiles > 1)
    embed_cross_kernel<<<dim3(tiles - 1, (d / 4 + 255) / 256), 256, 0, s>>>(
        w.keys, n_tok, tiles, d, w.piece, d_emb);
  return check_launch("aj_embed_bwd");
}
