// bfloat16 causal GQA attention over packed segments on v_mfma_f32_32x32x16_bf16.
//
// Orientation.  The 32x32 MFMA accumulator gives each lane one COLUMN and 16
// rows.  The forward and the dQ pass compute S^T = K Q^T so that a lane owns
// one query (a column) and holds 32 of the key scores of each 64-key tile: the
// online softmax is per lane plus one exchange with lane^32.  The probabilities
// then feed O^T = V^T P^T directly as the B operand: within one k-step a lane
// half contributes 8 keys, and the A operand (V^T, staged transposed in LDS)
// is read for exactly the same 8 keys, so the k order inside the instruction
// never has to match memory order.  The dK/dV pass computes S = Q K^T so that a
// lane owns one KEY, and accumulates dV^T = dO^T P and dK^T = Q^T dS the same
// way.  Segment masking: a query row attends to [segment start, itself].
//
// Workgroups: NW waves of 32 query (or key) rows each, all of them reading
// every staged tile, so that a tile copied into LDS serves 32 * NW rows.
// Query tiles are visited from the end of the pack (the longest rows first)
// and the head index varies fastest, so the query heads that share a
// key/value head run side by side.
#include "ops.h"

namespace aj {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;

AJ_DEV f32x16_t mfma(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

AJ_DEV uint32_t pack2(float lo, float hi) { return f2bf2(lo, hi); }

// 2^x on the hardware unit (v_exp_f32): the arguments here are <= 0 or -inf,
// where it needs none of exp2f's range handling.
AJ_DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// 8 accumulator values r0..r0+7 -> one bf16x8 operand
AJ_DEV bf16x8_t pack8(const f32x16_t &v, int r0) {
  u32x4_t u{pack2(v[r0], v[r0 + 1]), pack2(v[r0 + 2], v[r0 + 3]), pack2(v[r0 + 4], v[r0 + 5]),
            pack2(v[r0 + 6], v[r0 + 7])};
  return __builtin_bit_cast(bf16x8_t, u);
}

AJ_DEV int seg_of(const int32_t *cu, int n_seg, int base, int row) {
  int lo = 0, hi = n_seg - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (cu[mid] - base <= row) lo = mid; else hi = mid - 1;
  }
  return lo;
}
template <typename A> AJ_DEV int seg_start(const A &a, int row) {
  const int v = a.cu_seqlens[seg_of(a.cu_seqlens, a.n_seg, a.base, row)] - a.base;
  return v < 0 ? 0 : (v > row ? row : v);
}
template <typename A> AJ_DEV int seg_end(const A &a, int row) {
  const int v = a.cu_seqlens[seg_of(a.cu_seqlens, a.n_seg, a.base, row) + 1] - a.base;
  return v <= row ? row + 1 : (v > a.n_tok ? a.n_tok : v);
}

// Work item of workgroup wg: the items are ordered heaviest first (the last
// query tiles, or the first key tiles, of the pack), and the hardware deals
// workgroups round-robin to the 8 XCDs, so taking them in launch order gives
// every XCD an even share of the heavy and the light ones.  Dealing each XCD
// a contiguous range instead (for L2 locality) left the XCD holding the
// heaviest causal tiles of a 48k-token segment with ~1.75x the average work.
// Items are (tile, head) with the head fastest, so when the head count is a
// multiple of 8 every tile of a head still runs on one XCD.
AJ_DEV int work_item(int wg) { return wg; }

AJ_DEV float wave_min_f(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o, 64));
  return v;
}

// ------------------------------------------------------------------ LDS tiles
// A tile of 64 token rows x HD bfloat16, row-major in LDS (HD*2 bytes per
// row), filled by asynchronous direct-to-LDS copies (a wave instruction moves
// 64 x 16 bytes; lane l's bytes land at dst + 16*l).  Both fragment shapes
// read it:
//   row fragments (ds_read_b128): 32 consecutive tokens x 8 features, for the
//     products whose rows are tokens (S = Q K^T and its transposes);
//   column fragments (ds_read_b64_tr_b16): 32 consecutive features x 8
//     tokens, for the products whose rows are features (O^T = V^T P^T,
//     dQ^T = K^T dS^T, dV^T = dO^T P, dK^T = Q^T dS).
// 16-byte chunk c of token row r sits at chunk position c ^ swz(r).  With 64
// LDS banks (256 bytes a line), swz makes the 16 rows of a row read and the
// 4 rows x 2 chunks of a transposed read hit distinct bank groups:
//   HD = 128 (one row a line):  swz(r) = 2*(r & 7) | ((r >> 3) & 1)
//   HD = 64 (two rows a line):  swz(r) = 2*((r >> 1) & 3) | ((r >> 3) & 1)
// (bijective on 16 consecutive rows; within an aligned group of 4 rows the
// values differ in a bit other than bit 0, so chunks c and c^1 never meet).
constexpr int kTR = 64;       // token rows per staged tile

AJ_DEV uint32_t lds_addr(const void *p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}

template <int HD>
AJ_DEV int tok_swz(int r) {
  return HD == 128 ? ((r & 7) << 1) | ((r >> 3) & 1) : (((r >> 1) & 3) << 1) | ((r >> 3) & 1);
}

template <int HD, int NW = 4>
struct TokTile {
  static constexpr int CPR = HD / 8;                 // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;               // rows per 1 KB wave instruction
  static constexpr int kInstr = kTR * HD * 2 / 1024 / NW;  // per wave (NW waves)
  static_assert(kInstr >= 1 && kTR * HD * 2 / 1024 % NW == 0, "tile copy split");
  static constexpr int kHalfs = kTR * HD;
  static constexpr int kBytes = kHalfs * 2;

  AJ_DEV static int swz(int r) { return tok_swz<HD>(r); }
  // token rows [r0, r0 + 64) of `src` (row stride ld elements); rows at or
  // past `rows` copy row rows - 1 (their products are masked out).  tid is
  // the thread index (a caller short of registers passes it through an
  // opaque copy so that the per-lane offsets are recomputed, not kept live)
  AJ_DEV static void load(uint16_t *lds, const bf16_t *src, int64_t ld, int r0, int rows,
                          int tid = -1) {
    const int th = tid < 0 ? (int)threadIdx.x : tid;
    const int lane = th & 63, wave = th >> 6;
#pragma unroll
    for (int q = 0; q < kInstr; ++q) {
      const int blk = wave * kInstr + q;
      const int r = blk * RPI + lane / CPR;
      const int c = (lane % CPR) ^ swz(r);
      const int rr = min(r0 + r, rows - 1);
      __builtin_amdgcn_global_load_lds(src + (int64_t)rr * ld + 8 * c,
                                       (__attribute__((address_space(3))) void *)(lds + blk * 512),
                                       16, 0, 0);
    }
  }
};

// Per-lane LDS addresses of the fragment reads of TokTile tiles.  Every
// staged tile of a kernel sits at a fixed byte offset in one __shared__
// arena; a read passes that offset (plus its token row block's) as the
// instruction's immediate offset, so that a few address registers serve
// every tile, stage and row block.  The swizzle depends only on the token
// row mod 16 (row blocks start at multiples of 16), and a k-slice or a
// feature block enters the chunk index in bits that the lane's own part
// leaves free, so it is the lane's base XOR a constant.
template <int HD>
struct TileLanes {
  static constexpr int KS = HD / 16, DT = HD / 32, RB = HD * 2;   // RB: bytes per token row
  uint32_t row[KS];      // row fragment of k-slice kk
  uint32_t col[DT][2];   // column fragment of feature block i: token rows r and r + 8

  AJ_DEV void init(const void *arena) {
    const int lane = threadIdx.x & 63, l = lane & 31, hl = lane >> 5;
    const int g = lane >> 4, s = lane & 15;
    const uint32_t base = lds_addr(arena);
    // row fragments: token row l, chunk 2kk + hl
    const uint32_t rb = l * RB + 16 * (hl ^ tok_swz<HD>(l));
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) row[kk] = base + (rb ^ (32 * kk));
    // column fragments (ds_read_b64_tr_b16, see col_frag): source lane s of
    // 16-lane group g addresses token row r = 4(g/2) + s/4 and features
    // 32i + 16(g%2) + 4(s%4)..+3, i.e. chunk 4i + c0 at byte 8(s%2) in it;
    // row r + 8 has the swizzle of row r with bit 0 flipped
    const int r = 4 * (g >> 1) + (s >> 2), c0 = 2 * (g & 1) + ((s >> 1) & 1);
    const uint32_t cb = r * RB + 16 * (c0 ^ tok_swz<HD>(r)) + 8 * (s & 1);
#pragma unroll
    for (int i = 0; i < DT; ++i) {
      col[i][0] = base + (cb ^ (64 * i));
      col[i][1] = base + 8 * RB + (cb ^ (64 * i) ^ 16);
    }
  }
  // MFMA operand: rows = tokens [t0, t0 + 32) of the tile at byte offset off
  // (t0 * RB included in off), k = features [16kk, 16kk + 16)
  AJ_DEV bf16x8_t row_frag(const int off, const int kk) const {
    bf16x8_t v;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(row[kk]), "i"(off) : "memory");
    return v;
  }
  // MFMA operand: rows = features [32i, 32i + 32), k = 8 tokens in the order
  // the accumulator-to-operand packing (pack8) produces: lane half h holds
  // tokens t0 + 4h + 0..3 and t0 + 8 + 4h + 0..3 (t0 * RB included in off).
  // ds_read_b64_tr_b16: in a 16-lane group, lane j receives element j%4 of
  // the 4-element run addressed by lane 4e + j/4; source lane s addresses
  // token row t + s/4, features fb + 4*(s%4)..+3, so lane j receives feature
  // fb + j at 4 tokens.
  AJ_DEV bf16x8_t col_frag(const int off, const int i) const {
    u32x2_t lo, hi;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(lo) : "v"(col[i][0]), "i"(off) : "memory");
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(hi) : "v"(col[i][1]), "i"(off) : "memory");
    return __builtin_bit_cast(bf16x8_t, u32x4_t{lo[0], lo[1], hi[0], hi[1]});
  }
};

// Waits for every LDS read in flight; the operands pass through empty
// statements after the wait so that no MFMA consuming them moves above it.
template <int N>
AJ_DEV void lds_wait(bf16x8_t (&v)[N]) {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(v[i]));
}
AJ_DEV void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

typedef float f32x4_t __attribute__((ext_vector_type(4)));
// 4 consecutive floats from LDS at byte address a + off (inline assembly,
// like the fragment reads: the tile copies of the next item may still be in
// flight)
AJ_DEV f32x4_t lds_read_f4(const uint32_t a, const int off) {
  f32x4_t v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(a), "i"(off) : "memory");
  return v;
}
AJ_DEV void dma_wait() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Waits until at most n LDS reads (inline assembly, issued in order) are in
// flight (n a constant after inlining, 0..15).
AJ_DEV void lds_wait_n(int n) {
  switch (n) {
    case 1: asm volatile("s_waitcnt lgkmcnt(1)" ::: "memory"); break;
    case 2: asm volatile("s_waitcnt lgkmcnt(2)" ::: "memory"); break;
    case 3: asm volatile("s_waitcnt lgkmcnt(3)" ::: "memory"); break;
    case 4: asm volatile("s_waitcnt lgkmcnt(4)" ::: "memory"); break;
    case 5: asm volatile("s_waitcnt lgkmcnt(5)" ::: "memory"); break;
    case 6: asm volatile("s_waitcnt lgkmcnt(6)" ::: "memory"); break;
    case 7: asm volatile("s_waitcnt lgkmcnt(7)" ::: "memory"); break;
    case 8: asm volatile("s_waitcnt lgkmcnt(8)" ::: "memory"); break;
    case 9: asm volatile("s_waitcnt lgkmcnt(9)" ::: "memory"); break;
    case 10: asm volatile("s_waitcnt lgkmcnt(10)" ::: "memory"); break;
    case 11: asm volatile("s_waitcnt lgkmcnt(11)" ::: "memory"); break;
    case 12: asm volatile("s_waitcnt lgkmcnt(12)" ::: "memory"); break;
    case 13: asm volatile("s_waitcnt lgkmcnt(13)" ::: "memory"); break;
    case 14: asm volatile("s_waitcnt lgkmcnt(14)" ::: "memory"); break;
    default: asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); break;
  }
}

// acc[t] (t = 0, 1: token rows 32t..32t+31 of the tile at byte offset off)
// += tile rows x B, B = per-lane operands bv[kk] (k = features
// 16kk..16kk+15); with kZero the products start from zero (acc is not read:
// the first MFMA of each chain takes the constant 0 as its accumulator).
// Fragment q = 2kk + t feeds MFMA q and is read kAhead MFMAs ahead.
template <int HD, bool kZero = false>
AJ_DEV void rows_times(f32x16_t (&acc)[2], const TileLanes<HD> &L, const int off,
                       const bf16x8_t (&bv)[HD / 16]) {
  constexpr int KS = HD / 16, RB = HD * 2, NQ = 2 * KS, kAhead = 4;
  bf16x8_t f[NQ];
  auto read = [&](const int q) __attribute__((always_inline)) {
    f[q] = L.row_frag(off + (q & 1) * 32 * RB, q >> 1);
  };
#pragma unroll
  for (int q = 0; q < kAhead; ++q) read(q);
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    if (q + kAhead < NQ) read(q + kAhead);
    // one read per fragment; those issued after fragment q may stay in flight
    lds_wait_n((q + kAhead < NQ ? q + kAhead : NQ - 1) - q);
    asm volatile("" : "+v"(f[q]));
    const int kk = q >> 1, t = q & 1;
    const bool fresh = kZero && kk == 0;
    acc[t] = mfma(f[q], bv[kk], fresh ? f32x16_t{} : acc[t]);
  }
}

// acc[i] (features 32i..32i+31) += tile^T x P for the tile at byte offset
// off, P given per 16-token chunk j as packed accumulator halves pj[j]
// (tokens 32(j/2) + 16(j%2) + pack8 order).  Fragment q = j DT + i feeds
// MFMA q and is read kAhead MFMAs ahead (two LDS reads per fragment).
template <int HD>
AJ_DEV void cols_times(f32x16_t (&acc)[HD / 32], const TileLanes<HD> &L, const int off,
                       const bf16x8_t (&pj)[4]) {
  constexpr int DT = HD / 32, RB = HD * 2, NQ = 4 * DT, kAhead = 4;
  bf16x8_t f[NQ];
  auto read = [&](const int q) __attribute__((always_inline)) {
    const int j = q / DT;
    f[q] = L.col_frag(off + (32 * (j >> 1) + 16 * (j & 1)) * RB, q % DT);
  };
#pragma unroll
  for (int q = 0; q < kAhead; ++q) read(q);
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    if (q + kAhead < NQ) read(q + kAhead);
    lds_wait_n(2 * ((q + kAhead < NQ ? q + kAhead : NQ - 1) - q));
    asm volatile("" : "+v"(f[q]));
    acc[q % DT] = mfma(f[q], pj[q / DT], acc[q % DT]);
  }
}

// A workgroup barrier without the memory fence of __syncthreads (which would
// also wait for every LDS read and copy in flight); the waits it needs are
// explicit before it, and the empty statements keep the compiler from moving
// memory operations across it.
AJ_DEV void bar_nofence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// One 32-row block (token rows t0..t0+31) of two staged tiles, at byte
// offsets offa and offb, against the lane's operands: sa = ta rows x ka,
// sb = sb0 + tb rows x kb (k = features; the incoming sa, sb are not read).
// Fragments are read two k-steps ahead; each step waits only for its own.
template <int HD>
AJ_DEV void rows_times_pair(f32x16_t &sa, f32x16_t &sb, const TileLanes<HD> &L, const int offa,
                            const int offb, const int t0, const bf16x8_t (&ka)[HD / 16],
                            const bf16x8_t (&kb)[HD / 16], const f32x16_t &sb0) {
  constexpr int KS = HD / 16, RB = HD * 2;
  bf16x8_t fa[KS], fb[KS];
#pragma unroll
  for (int kk = 0; kk < 2 && kk < KS; ++kk) {
    fa[kk] = L.row_frag(offa + t0 * RB, kk);
    fb[kk] = L.row_frag(offb + t0 * RB, kk);
  }
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    if (kk + 2 < KS) {
      fa[kk + 2] = L.row_frag(offa + t0 * RB, kk + 2);
      fb[kk + 2] = L.row_frag(offb + t0 * RB, kk + 2);
    }
    // reads issued after this step's pair: those of steps kk+1 .. min(kk+2, KS-1)
    lds_wait_n(2 * ((kk + 2 < KS ? kk + 2 : KS - 1) - kk));
    asm volatile("" : "+v"(fa[kk]));
    asm volatile("" : "+v"(fb[kk]));
    sa = mfma(fa[kk], ka[kk], kk == 0 ? f32x16_t{} : sa);
    sb = mfma(fb[kk], kb[kk], kk == 0 ? sb0 : sb);
  }
}

// acc[i] (features 32i..32i+31) += tile^T x P over tokens t0..t0+31 of the
// tile at byte offset off, P given as the two packed accumulator halves of
// that 32-row block (pack8 order).  Fragment q = 2i + h (token rows
// t0 + 16h) feeds MFMA q and is read kAhead MFMAs ahead.
template <int HD>
AJ_DEV void cols_times_half(f32x16_t (&acc)[HD / 32], const TileLanes<HD> &L, const int off,
                            const int t0, const bf16x8_t (&pj)[2]) {
  constexpr int DT = HD / 32, RB = HD * 2, NQ = 2 * DT, kAhead = 3;
  bf16x8_t f[NQ];
  auto read = [&](const int q) __attribute__((always_inline)) {
    f[q] = L.col_frag(off + (t0 + 16 * (q & 1)) * RB, q >> 1);
  };
#pragma unroll
  for (int q = 0; q < kAhead && q < NQ; ++q) read(q);
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    if (q + kAhead < NQ) read(q + kAhead);
    lds_wait_n(2 * ((q + kAhead < NQ ? q + kAhead : NQ - 1) - q));
    asm volatile("" : "+v"(f[q]));
    acc[q >> 1] = mfma(f[q], pj[q & 1], acc[q >> 1]);
  }
}

// ------------------------------------------------------------------ forward
// One workgroup: 32 * NW queries of one head (NW waves of 32), key tiles of 64
// double-buffered and shared by all the waves; a lane owns one query.
template <int HD, int NW>
__global__ __launch_bounds__(64 * NW, 2) void attn_fwd_mfma_kernel(AttnArgs a, int n_qt) {
  using TT = TokTile<HD, NW>;
  constexpr int KS = HD / 16, DT = HD / 32, T = TT::kBytes;
  // two stages of a K and a V tile: K at 0 and T, V at 2T and 3T (bytes)
  __shared__ __attribute__((aligned(16))) uint16_t sm[4 * TT::kHalfs];
  __shared__ int rng[2];
  TileLanes<HD> L;
  L.init(sm);
  const int t = work_item(blockIdx.x);
  const int h = t % a.Hq, qt = n_qt - 1 - t / a.Hq;
  const int g = (h * a.Hkv) / a.Hq;
  const int ld = (a.Hq + 2 * a.Hkv) * HD;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hl = lane >> 5, lq = lane & 31;
  const int q0 = qt * 32 * NW;
  const int q = q0 + 32 * w + lq;
  const bool qv = q < a.n_tok;
  const int qs = qv ? seg_start(a, q) : a.n_tok;
  const bf16_t *qkv = (const bf16_t *)a.qkv;
  if (threadIdx.x == 0) {
    rng[0] = seg_start(a, q0);
    rng[1] = min(q0 + 32 * NW - 1, a.n_tok - 1);
  }
  bf16x8_t qf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    u32x4_t x{0, 0, 0, 0};
    if (qv) x = *(const u32x4_t *)(qkv + (int64_t)q * ld + h * HD + 16 * kk + 8 * hl);
    qf[kk] = __builtin_bit_cast(bf16x8_t, x);
  }
  f32x16_t o[DT];
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[i][r] = 0.f;
  float m = -INFINITY, lsum = 0.f;
  const float c = a.scale * kLog2e;
  const int w_lo = (int)wave_min_f((float)qs);          // earliest key any row of the wave reads
  const int w_hi = min(q0 + 32 * w + 31, a.n_tok - 1);   // latest query row of the wave
  const int w_qs = (int)-wave_min_f(-(float)qs);        // latest segment start of the wave
  __syncthreads();
  const int kv_lo = rng[0], kv_hi = rng[1];
  const int n_kt = (kv_hi - kv_lo + kTR) / kTR;
  const bf16_t *kbase = qkv + (a.Hq + g) * HD, *vbase = qkv + (a.Hq + a.Hkv + g) * HD;
  TT::load(sm, kbase, ld, kv_lo, kv_hi + 1);
  TT::load(sm + 2 * TT::kHalfs, vbase, ld, kv_lo, kv_hi + 1);
  dma_wait();
  __syncthreads();
  // tile it reads stage st and prefetches tile it + 1 into the other stage;
  // the loop runs two tiles per pass so that both stages are fixed offsets
  auto tile = [&](const int it, const int st) __attribute__((always_inline)) {
    const int k0 = kv_lo + it * kTR;
    if (it + 1 < n_kt) {
      TT::load(sm + (st ^ 1) * TT::kHalfs, kbase, ld, k0 + kTR, kv_hi + 1);
      TT::load(sm + (2 + (st ^ 1)) * TT::kHalfs, vbase, ld, k0 + kTR, kv_hi + 1);
    }
    if (k0 <= w_hi && k0 + kTR - 1 >= w_lo) {
      f32x16_t s[2];
      rows_times<HD, true>(s, L, st * T, qf);            // S^T = K Q^T (unscaled)
      float mx = -INFINITY;
      if (k0 >= w_qs && k0 + kTR - 1 <= q0 + 32 * w) {   // every key visible to every row
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[tt][r]);
      } else {
        const int lo = qs - k0 - 4 * hl, hi = q - k0 - 4 * hl;
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int off = 32 * tt + 8 * (r >> 2) + (r & 3);
            s[tt][r] = (off >= lo && off <= hi) ? s[tt][r] : -INFINITY;
            mx = fmaxf(mx, s[tt][r]);
          }
      }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64)) * c;        // log2 units (c > 0)
      // The running maximum m moves only when a row's tile maximum exceeds it
      // by more than 8 (log2 units): the weights exp2(s c - m) then stay
      // below 2^8, and the rescale of O and the sum runs, for the whole wave,
      // only when some row needs it.  m is the same stale value in the final
      // log-sum-exp, so the result is exact.
      const bool grow = mx > m + 8.f;                      // also when m is still -inf
      if (__builtin_amdgcn_ballot_w64(grow)) {
        const float mn = grow ? mx : m;
        const float alpha = grow ? fast_exp2(m - mn) : 1.f;   // 0 when m was -inf
#pragma unroll
        for (int i = 0; i < DT; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[i][r] *= alpha;
        lsum *= alpha;
        m = mn;
      }
      // m is -inf only while every score the row has seen is -inf (masked):
      // then exp2(-inf + 0) = 0 without a select per score.  lsum holds this
      // lane half's keys only (both halves share m); the halves are added
      // once, after the last tile.
      const float nm = m == -INFINITY ? 0.f : -m;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = fast_exp2(fmaf(s[tt][r], c, nm));
          s[tt][r] = p;
          lsum += p;
        }
      const bf16x8_t pj[4] = {pack8(s[0], 0), pack8(s[0], 8), pack8(s[1], 0), pack8(s[1], 8)};
      cols_times<HD>(o, L, (2 + st) * T, pj);            // O^T += V^T P^T
    }
    lds_wait();
    dma_wait();
    __syncthreads();
  };
  for (int it = 0; it < n_kt; it += 2) {
    tile(it, 0);
    if (it + 1 < n_kt) tile(it + 1, 1);
  }
  lsum += __shfl_xor(lsum, 32, 64);
  if (!qv) return;
  const float inv = 1.f / lsum;
  bf16_t *out = (bf16_t *)a.o + (int64_t)q * a.Hq * HD + h * HD;
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int d = 32 * i + 8 * r4 + 4 * hl;
      *(u32x2_t *)(out + d) = u32x2_t{pack2(o[i][4 * r4] * inv, o[i][4 * r4 + 1] * inv),
                                      pack2(o[i][4 * r4 + 2] * inv, o[i][4 * r4 + 3] * inv)};
    }
  // log-sum-exp of the scaled scores in log2 units (the backward passes
  // work in exp2): log2(sum exp2(s c)) = m + log2(lsum)
  if (hl == 0) a.lse[(int64_t)h * a.n_tok + q] = m + log2f(lsum);
}

// ------------------------------------------------------------------ dQ
// Same workgroup shape as the forward; a lane owns one query.
template <int HD, int NW>
__global__ __launch_bounds__(64 * NW, 2) void attn_dq_mfma_kernel(AttnBwdArgs a, int n_qt) {
  using TT = TokTile<HD, NW>;
  constexpr int KS = HD / 16, DT = HD / 32, T = TT::kBytes;
  // two stages of a K and a V tile: K at 0 and T, V at 2T and 3T (bytes)
  __shared__ __attribute__((aligned(16))) uint16_t sm[4 * TT::kHalfs];
  __shared__ int rng[2];
  TileLanes<HD> L;
  L.init(sm);
  const int t = work_item(blockIdx.x);
  const int h = t % a.Hq, qt = n_qt - 1 - t / a.Hq;
  const int g = (h * a.Hkv) / a.Hq;
  const int ld = (a.Hq + 2 * a.Hkv) * HD;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hl = lane >> 5, lq = lane & 31;
  const int q0 = qt * 32 * NW;
  const int q = q0 + 32 * w + lq;
  const bool qv = q < a.n_tok;
  const int qs = qv ? seg_start(a, q) : a.n_tok;
  const bf16_t *qkv = (const bf16_t *)a.qkv;
  const bf16_t *dout = (const bf16_t *)a.dout;
  if (threadIdx.x == 0) {
    rng[0] = seg_start(a, q0);
    rng[1] = min(q0 + 32 * NW - 1, a.n_tok - 1);
  }
  bf16x8_t qf[KS], df[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    u32x4_t x{0, 0, 0, 0}, y{0, 0, 0, 0};
    if (qv) {
      x = *(const u32x4_t *)(qkv + (int64_t)q * ld + h * HD + 16 * kk + 8 * hl);
      y = *(const u32x4_t *)(dout + (int64_t)q * a.Hq * HD + h * HD + 16 * kk + 8 * hl);
    }
    qf[kk] = __builtin_bit_cast(bf16x8_t, x);
    df[kk] = __builtin_bit_cast(bf16x8_t, y);
  }
  const float lse2 = qv ? a.lse[(int64_t)h * a.n_tok + q] : 0.f;       // log2 units
  // the lane's query keeps one negated delta: every dP^T element starts from it
  const float ndlt = qv ? a.delta[(int64_t)h * a.n_tok + q] : 0.f;
  f32x16_t dp0;
#pragma unroll
  for (int r = 0; r < 16; ++r) dp0[r] = ndlt;
  f32x16_t acc[DT];
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
  const float c = a.scale * kLog2e;
  const int w_lo = (int)wave_min_f((float)qs);
  const int w_hi = min(q0 + 32 * w + 31, a.n_tok - 1);
  const int w_qs = (int)-wave_min_f(-(float)qs);        // latest segment start of the wave
  __syncthreads();
  const int kv_lo = rng[0], kv_hi = rng[1];
  const int n_kt = (kv_hi - kv_lo + kTR) / kTR;
  const bf16_t *kbase = qkv + (a.Hq + g) * HD, *vbase = qkv + (a.Hq + a.Hkv + g) * HD;
  TT::load(sm, kbase, ld, kv_lo, kv_hi + 1);
  TT::load(sm + 2 * TT::kHalfs, vbase, ld, kv_lo, kv_hi + 1);
  dma_wait();
  __syncthreads();
  // key rows 32tt..32tt+31 of the tile at stage st: S^T = K Q^T, dP^T =
  // V dO^T, the softmax terms, then dQ^T += K^T dS^T over those 32 keys
  auto half = [&](const int tt, const int st, const int k0,
                  const bool full) __attribute__((always_inline)) {
    f32x16_t s, dp;   // S^T and dP^T - delta, set by rows_times_pair
    rows_times_pair<HD>(s, dp, L, st * T, (2 + st) * T, 32 * tt, qf, df, dp0);
    if (full) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = fast_exp2(fmaf(s[r], c, -lse2)) * dp[r];
    } else {
      // key k0 + 4hl + off (off a constant per element) is visible iff
      // lo <= off <= hi
      const int lo = qs - k0 - 4 * hl, hi = q - k0 - 4 * hl;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int off = 32 * tt + 8 * (r >> 2) + (r & 3);
        const float p = (off >= lo && off <= hi) ? fast_exp2(fmaf(s[r], c, -lse2)) : 0.f;
        s[r] = p * dp[r];
      }
    }
    const bf16x8_t sj[2] = {pack8(s, 0), pack8(s, 8)};
    cols_times_half<HD>(acc, L, st * T, 32 * tt, sj);   // dQ^T += K^T dS^T
  };
  // tile it reads stage st and prefetches tile it + 1 into the other stage;
  // two tiles per pass so that both stages are fixed offsets
  auto tile = [&](const int it, const int st) __attribute__((always_inline)) {
    const int k0 = kv_lo + it * kTR;
    if (it + 1 < n_kt) {
      TT::load(sm + (st ^ 1) * TT::kHalfs, kbase, ld, k0 + kTR, kv_hi + 1);
      TT::load(sm + (2 + (st ^ 1)) * TT::kHalfs, vbase, ld, k0 + kTR, kv_hi + 1);
    }
    if (k0 <= w_hi && k0 + kTR - 1 >= w_lo) {
      const bool full = k0 >= w_qs && k0 + kTR - 1 <= q0 + 32 * w;   // every key visible to every row
      half(0, st, k0, full);
      half(1, st, k0, full);
    }
    lds_wait();
    dma_wait();
    __syncthreads();
  };
  for (int it = 0; it < n_kt; it += 2) {
    tile(it, 0);
    if (it + 1 < n_kt) tile(it + 1, 1);
  }
  if (!qv) return;
  bf16_t *out = (bf16_t *)a.dqkv + (int64_t)q * ld + h * HD;
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int d = 32 * i + 8 * r4 + 4 * hl;
      *(u32x2_t *)(out + d) = u32x2_t{pack2(acc[i][4 * r4] * a.scale, acc[i][4 * r4 + 1] * a.scale),
                                      pack2(acc[i][4 * r4 + 2] * a.scale, acc[i][4 * r4 + 3] * a.scale)};
    }
}

// ------------------------------------------------------------------ dK, dV
// One workgroup: 32 * NW keys of one key/value head (NW waves of 32), a lane
// owns one key; it walks every query head of the group and the segment's
// query tiles of 64 after the keys (items), staged three deep (Q, dO and the
// queries' LSE and delta) and shared by all the waves.
//
// A lane holds its key's K and V rows and its dK, dV accumulators, which
// leaves room for one wave per SIMD: nothing else on the SIMD covers the
// wave's waits, so each wave runs a software pipeline over the items'
// 32-query halves u.  Step u first issues, one MFMA at a time, the products
// dV^T += dO^T P and dK^T += Q^T dS of half u - 1 and, between them, the
// vector work of half u's softmax terms (exponentials, masks, bf16 packing of
// P and dS); then the products S = Q K^T and dP - delta = dO V^T - delta of
// half u + 1 (its dP accumulators start from the half's negated delta) into
// the same registers.  The LDS reads of the fragments run a few MFMAs ahead,
// and those of half u + 1's LSE one step ahead of its softmax.

template <int V> struct Ci { static constexpr int value = V; };

// fn(Ci<I>{}) for I = B..E-1, each call with its index as a constant
template <int B, int E>
struct StaticFor {
  template <typename Fn> AJ_DEV static void run(Fn &fn) {
    fn(Ci<B>{});
    StaticFor<B + 1, E>::run(fn);
  }
};
template <int E>
struct StaticFor<E, E> {
  template <typename Fn> AJ_DEV static void run(Fn &) {}
};

// LDS read schedule of one step: NS MFMA slots, the first NC = NS / 2 the
// dV/dK products (fragment: two ds_read_b64_tr_b16), the rest the S/dP
// products (fragment: one ds_read_b128).  Fragment j (the operand of MFMA j)
// is read D slots ahead, so a step begins with its fragments 0..D-1 in
// flight (read by the step before, after the LSE and delta of the step's
// softmax half).  After slot NC the step reads the next half's LSE and delta
// (8 reads).  In a step with a barrier between the two groups (the next
// item's tile becomes visible there), the S/dP fragments are read after it.
template <int NS, int D>
struct DkvSched {
  static constexpr int NC = NS / 2;
  static constexpr int size(int f) { return f % NS < NC ? 2 : 1; }   // f >= NS: next step's
  // fragments [first, last) read after slot s
  static constexpr int first(int s, bool bar) {
    return bar && s < NC - 1 && s + D >= NC ? 0 : bar && s == NC - 1 ? NC : s + D;
  }
  static constexpr int last(int s, bool bar) {
    return bar && s < NC - 1 && s + D >= NC ? 0 : bar && s == NC - 1 ? NC + D : s + D + 1;
  }
  // LDS reads still allowed in flight when MFMA j waits for its fragment
  static constexpr int wait(int j, bool bar) {
    int cnt = 0, end = -1;
    for (int f = 0; f < D; ++f) {
      cnt += size(f);
      if (f == j) end = cnt;
    }
    for (int s = 0; s < j; ++s) {
      for (int f = first(s, bar); f < last(s, bar); ++f) {
        cnt += size(f);
        if (f == j) end = cnt;
      }
      if (s == NC) cnt += 8;
    }
    return cnt - end;
  }
  // slot of the vector work of softmax score r (0..15): spread over the
  // dV/dK group (the LSE was read before fragment 0)
  static constexpr int score_slot(int r) { return r * NC / 16; }
  // Order of the S/dP group's products (KS k-slices each): position u is S
  // (Q fragment) or dP (dO fragment) of k-slice kk(u).  The first dP product
  // comes at u = 4: its accumulator starts from the half's negated delta,
  // read from LDS right after the group's first MFMA, so fragment 4's reads,
  // issued after the delta's, have landed by then and the delta with them
  // (LDS returns in order).  S and dP alternate after that, so that few
  // products wait on the one before.
  static constexpr int KS = NS / 4;
  static_assert(KS >= 4, "the first dP product at position 4");
  static constexpr bool is_s(int u) { return u < 4 || (u - 4 < 2 * (KS - 4) && ((u - 4) & 1)); }
  static constexpr int kk(int u) {
    return u < 4 ? u
           : u - 4 < 2 * (KS - 4) ? (((u - 4) & 1) ? 4 + (u - 4) / 2 : (u - 4) / 2)
                                  : u - 4 - (KS - 4);
  }
};

template <int HD, int NW>
__global__ __launch_bounds__(64 * NW) void attn_dkv_mfma_kernel(AttnBwdArgs a, int /*n_kt*/) {
  using TT = TokTile<HD, NW>;
  constexpr int KS = HD / 16, DT = HD / 32, T = TT::kBytes, RB = HD * 2;
  constexpr int NS = 8 * DT, NC = NS / 2, D = 3;
  using Sched = DkvSched<NS, D>;
  static_assert(Sched::wait(0, false) <= 15 && Sched::wait(NC + 1, false) <= 15, "lgkmcnt range");
  // three stages of a Q tile (region smq) and a dO tile (region smd) at s*T;
  // the stages' LSE (rows 0..2) and delta (rows 3..5)
  __shared__ __attribute__((aligned(16))) uint16_t smq[3 * TT::kHalfs];
  __shared__ __attribute__((aligned(16))) uint16_t smd[3 * TT::kHalfs];
  __shared__ __attribute__((aligned(16))) float ld_sm[6][kTR];
  __shared__ int rng[1];
  TileLanes<HD> LQ, LD;
  LQ.init(smq);
  LD.init(smd);
  const int t = work_item(blockIdx.x);
  const int g = t % a.Hkv, kt = t / a.Hkv;   // early keys of a segment see the most queries
  const int ld = (a.Hq + 2 * a.Hkv) * HD;
  const int ldo = a.Hq * HD;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hl = lane >> 5, lq = lane & 31;
  const int k0 = kt * 32 * NW;
  const int kv = k0 + 32 * w + lq;            // the key row this lane owns
  const bool kvv = kv < a.n_tok;
  const int ke = kvv ? seg_end(a, kv) : 0;    // queries of the key: [kv, ke)
  const bf16_t *qkv = (const bf16_t *)a.qkv;
  const bf16_t *dout = (const bf16_t *)a.dout;
  if (threadIdx.x == 0) rng[0] = seg_end(a, min(k0 + 32 * NW - 1, a.n_tok - 1));
  bf16x8_t kf[KS], vf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    u32x4_t x{0, 0, 0, 0}, y{0, 0, 0, 0};
    if (kvv) {
      x = *(const u32x4_t *)(qkv + (int64_t)kv * ld + (a.Hq + g) * HD + 16 * kk + 8 * hl);
      y = *(const u32x4_t *)(qkv + (int64_t)kv * ld + (a.Hq + a.Hkv + g) * HD + 16 * kk + 8 * hl);
    }
    kf[kk] = __builtin_bit_cast(bf16x8_t, x);
    vf[kk] = __builtin_bit_cast(bf16x8_t, y);
    // the key and value rows are only ever MFMA operands: keep them in the
    // accumulation registers (the vector registers are the scarce ones)
    asm volatile("" : "+a"(kf[kk]));
    asm volatile("" : "+a"(vf[kk]));
  }
  f32x16_t dk[DT], dv[DT];
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) { dk[i][r] = 0.f; dv[i][r] = 0.f; }
  const float c = a.scale * kLog2e;
  // The products of half -1 (the first step's dV/dK group) read stage 2 with
  // zero P and dS: clear it so that they add exact zeros.
  {
    const u32x4_t z{0, 0, 0, 0};
    for (int i = threadIdx.x; i < TT::kHalfs / 8; i += 64 * NW) {
      *(u32x4_t *)(smq + 2 * TT::kHalfs + 8 * i) = z;
      *(u32x4_t *)(smd + 2 * TT::kHalfs + 8 * i) = z;
    }
  }
  __syncthreads();
  const int q_hi = rng[0];    // queries [k0, q_hi)
  const int group = a.Hq / a.Hkv;
  const int n_qb = q_hi > k0 ? (q_hi - k0 + kTR - 1) / kTR : 0;
  const int n_it = group * n_qb;
  // item it: query head g*group + it / n_qb, query tile k0 + 64 * (it % n_qb)
  auto load_item = [&](int it, auto ST) __attribute__((always_inline)) {
    constexpr int st = decltype(ST)::value;
    const int h = g * group + it / n_qb, qb = k0 + kTR * (it % n_qb);
    TT::load(smq + st * TT::kHalfs, qkv + h * HD, ld, qb, q_hi);
    TT::load(smd + st * TT::kHalfs, dout + h * HD, ldo, qb, q_hi);
    if (w < 2) {                // one float per lane: LSE (wave 0), delta (wave 1)
      const float *src = (w == 0 ? a.lse : a.delta) + (int64_t)h * a.n_tok + min(qb + lane, q_hi - 1);
      __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)ld_sm[3 * w + st],
                                       4, 0, 0);
    }
  };
  // the lane's LSE / delta reads: 4 floats at 16 hl bytes past the offset
  const uint32_t ld_lane = lds_addr(ld_sm) + 16 * hl;

  // pipeline state: S, dP - delta of the current half (s, dp: exponentiated
  // in a step's first group, overwritten by the next half's products in its
  // second); that half's LSE (lv) and the next half's negated delta (dl, the
  // initial value of its dP); packed P, dS of the previous half (pp, sp) and
  // of the current one (pc, spc)
  f32x16_t s, dp;
  f32x4_t lv[4], dl[4];
  bf16x8_t pp[2], sp[2], pc[2], spc[2];
  const bf16x8_t zero8 = __builtin_bit_cast(bf16x8_t, u32x4_t{0, 0, 0, 0});
  pp[0] = pp[1] = sp[0] = sp[1] = zero8;
  pc[0] = pc[1] = spc[0] = spc[1] = zero8;
  // LSE (log2 units) and delta of the lane's 16 query rows of half (tt, st):
  // 32tt + 8(r/4) + 4hl + r%4
  auto read_ld = [&](const int tt, const int st) __attribute__((always_inline)) {
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      lv[r4] = lds_read_f4(ld_lane, st * 256 + (32 * tt + 8 * r4) * 4);
      dl[r4] = lds_read_f4(ld_lane, (3 + st) * 256 + (32 * tt + 8 * r4) * 4);
    }
  };
  // the negated delta of the lane's 16 query rows as an accumulator
  auto delta_init = [&]() __attribute__((always_inline)) -> f32x16_t {
    f32x16_t v;
#pragma unroll
    for (int r = 0; r < 16; ++r) v[r] = dl[r >> 2][r & 3];
    return v;
  };

  // fragment j of a step: dV/dK group (j < NC): dv[i] (j < NC/2, dO tile) or
  // dk[i] (Q tile), feature block i = j % DT, token rows 32tt + 16((j/DT)%2);
  // S/dP group: k-slice Sched::kk(j - NC) of the Q or dO tile rows 32tt
  auto read_frag = [&](const int j, const int tt_c, const int st_c, const int tt_p,
                       const int st_p) __attribute__((always_inline)) -> bf16x8_t {
    if (j < NC) {
      const int i = j % DT, hb = (j / DT) & 1;
      const int off = st_c * T + (32 * tt_c + 16 * hb) * RB;
      return j < NC / 2 ? LD.col_frag(off, i) : LQ.col_frag(off, i);
    }
    const int off = st_p * T + 32 * tt_p * RB;
    return Sched::is_s(j - NC) ? LQ.row_frag(off, Sched::kk(j - NC))
                               : LD.row_frag(off, Sched::kk(j - NC));
  };

  // The causal and segment mask enters S as its accumulator's initial value:
  // 0 where the lane's key sees the query row, -inf where it does not (then
  // P = exp2(-inf) = 0 and dS = 0).  Most halves are seen whole by every
  // lane of the wave and start from 0; only the others build the bias.
  // Query row offset o (past 4hl) of a half is seen iff
  // (unsigned)(o - lo) < span.
  auto seen_whole = [&](const int lo, const int span) __attribute__((always_inline)) {
    return __builtin_amdgcn_ballot_w64(!(lo <= 0 && 27 - lo < span)) == 0;
  };
  // first S product of a half: F Q-fragment, K-slice 0
  auto s_first = [&](const bf16x8_t &fq, const bool whole, const int lo,
                     const int span) __attribute__((always_inline)) -> f32x16_t {
    if (whole) return mfma(fq, kf[0], f32x16_t{});
    f32x16_t bias;
#pragma unroll
    for (int r = 0; r < 16; ++r)
      bias[r] = (uint32_t)(8 * (r >> 2) + (r & 3) - lo) < (uint32_t)span ? 0.f : -INFINITY;
    return mfma(fq, kf[0], bias);
  };

  bf16x8_t F[NS];
  // One step: dV/dK products of half (tt_c, st_c) with pp, sp while the
  // softmax terms of the current half (s, dp, lv, dl) go into pc, spc; then
  // the S/dP products of half (tt_p, st_p), masked by (lo_p, span_p), into
  // s, dp, and that half's LSE and delta into lv, dl.  On entry F[0..D-1]
  // are in flight, on exit the next step's (its dV/dK group: half
  // (tt_s, st_s), this step's softmax half).  With BAR, a barrier between
  // the groups makes the next item's stage visible, then `after` runs.
  auto step = [&](auto TTC, auto STC, auto TTS, auto STS, auto TTP, auto STP, auto BAR,
                  const int lo_p, const int span_p, auto after) __attribute__((always_inline)) {
    constexpr int tt_c = decltype(TTC)::value, st_c = decltype(STC)::value;
    constexpr int tt_s = decltype(TTS)::value, st_s = decltype(STS)::value;
    constexpr int tt_p = decltype(TTP)::value, st_p = decltype(STP)::value;
    constexpr bool bar = decltype(BAR)::value != 0;
    const bool whole_p = seen_whole(lo_p, span_p);
    float pv[16], dq[16];
    auto slot = [&](auto JC) __attribute__((always_inline)) {
      constexpr int j = decltype(JC)::value;
      constexpr int wn = Sched::wait(j, bar);
      constexpr int f0 = Sched::first(j, bar), f1 = Sched::last(j, bar);
      lds_wait_n(wn);
      asm volatile("" : "+v"(F[j]));
      if (j == 0) {
        // the LSE reads precede fragment 0
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) asm volatile("" : "+v"(lv[r4]));
      }
      if (j < NC) {
        const int i = j % DT, hb = (j / DT) & 1;
        if (j < NC / 2) dv[i] = mfma(F[j], pp[hb], dv[i]);   // dV^T += dO^T P
        else dk[i] = mfma(F[j], sp[hb], dk[i]);              // dK^T += Q^T dS
      } else {
        constexpr int kk = Sched::kk(j - NC);
        if constexpr (Sched::is_s(j - NC)) {   // S = Q K^T (+ mask)
          s = kk == 0 ? s_first(F[j], whole_p, lo_p, span_p) : mfma(F[j], kf[kk], s);
        } else if constexpr (kk == 0) {    // dP - delta = dO V^T - delta
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4) asm volatile("" : "+v"(dl[r4]));
          dp = mfma(F[j], vf[0], delta_init());
        } else {
          dp = mfma(F[j], vf[kk], dp);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      if (bar && j == NC - 1) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        bar_nofence();
        after();
      }
#pragma unroll
      for (int f = f0; f < f1; ++f) {
        if (f < NS) F[f] = read_frag(f, tt_c, st_c, tt_p, st_p);
        else F[f - NS] = read_frag(f - NS, tt_s, st_s, 0, 0);
      }
      if (j == NC) read_ld(tt_p, st_p);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if (j >= NC || Sched::score_slot(r) != j) continue;
        // the score's inputs and the packed words pass through empty
        // statements, which keep this vector work in its slot (between the
        // slot's LDS reads and the next slot's wait) instead of gathered
        float sr = s[r], dr = dp[r];
        asm volatile("" : "+v"(sr), "+v"(dr));
        const float pr = fast_exp2(fmaf(sr, c, -lv[r >> 2][r & 3]));
        pv[r] = pr;
        dq[r] = pr * dr;
        if (r & 1) {
          const int h8 = r >> 3, k = (r & 7) >> 1;
          // the pair (r - 1, r) is word k of the packed half h8
          uint32_t wp = pack2(pv[r - 1], pv[r]), ws = pack2(dq[r - 1], dq[r]);
          asm volatile("" : "+v"(wp), "+v"(ws));
          u32x4_t up = __builtin_bit_cast(u32x4_t, pc[h8]);
          u32x4_t us = __builtin_bit_cast(u32x4_t, spc[h8]);
          up[k] = wp;
          us[k] = ws;
          pc[h8] = __builtin_bit_cast(bf16x8_t, up);
          spc[h8] = __builtin_bit_cast(bf16x8_t, us);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    };
    StaticFor<0, NS>::run(slot);
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      pp[x] = pc[x];
      sp[x] = spc[x];
    }
  };

  // One item (query tile of 64, two halves) at stage ST: the even step
  // exponentiates its first half, the odd one its second and, past the
  // barrier, stages item it + 2 into the stage item it - 1 used.  The loop
  // runs whole groups of three items (one per stage, so that every stage
  // offset is a constant and the loop has a single exit); the items past
  // n_it stage a copy of the last one and see no query (their P and dS are
  // zero, so their products add exact zeros).
  const int span = kvv ? ke - kv : 0;   // the key sees query rows [kv, ke)
  const int n_it3 = (n_it + 2) / 3 * 3;
  auto item = [&](const int it, auto ST) __attribute__((always_inline)) {
    constexpr int st = decltype(ST)::value;
    // half tt of item i: row offset o is seen iff o - (lo(i) - 32tt) < span(i)
    const int lo = kv - (k0 + kTR * (min(it, n_it - 1) % n_qb)) - 4 * hl;
    const int lo1 = kv - (k0 + kTR * (min(it + 1, n_it - 1) % n_qb)) - 4 * hl;
    step(Ci<1>{}, Ci<(st + 2) % 3>{}, Ci<0>{}, Ci<st>{}, Ci<1>{}, Ci<st>{}, Ci<0>{}, lo - 32,
         it < n_it ? span : 0, [] {});
    step(Ci<0>{}, Ci<st>{}, Ci<1>{}, Ci<st>{}, Ci<0>{}, Ci<(st + 1) % 3>{}, Ci<1>{}, lo1,
         it + 1 < n_it ? span : 0, [&]() __attribute__((always_inline)) {
           if (it + 2 < n_it3) load_item(min(it + 2, n_it - 1), Ci<(st + 2) % 3>{});
         });
  };
  // the last half's dV/dK products (its first D fragments are in flight)
  auto tail = [&](auto ST) __attribute__((always_inline)) {
    constexpr int st = decltype(ST)::value;
#pragma unroll
    for (int j = D; j < NC; ++j) F[j] = read_frag(j, 1, st, 0, 0);
    lds_wait();
#pragma unroll
    for (int j = 0; j < NC; ++j) {
      asm volatile("" : "+v"(F[j]));
      const int i = j % DT, hb = (j / DT) & 1;
      if (j < NC / 2) dv[i] = mfma(F[j], pp[hb], dv[i]);
      else dk[i] = mfma(F[j], sp[hb], dk[i]);
    }
  };
  if (n_it > 0) {
    load_item(0, Ci<0>{});
    load_item(min(1, n_it - 1), Ci<1>{});
    dma_wait();
    __syncthreads();
    // LSE and delta, then S and dP - delta of half 0
    const bool whole0 = seen_whole(kv - k0 - 4 * hl, span);
    read_ld(0, 0);
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      bf16x8_t fq = LQ.row_frag(0, kk), fd = LD.row_frag(0, kk);
      lds_wait();
      asm volatile("" : "+v"(fq));
      asm volatile("" : "+v"(fd));
      if (kk == 0) {
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) asm volatile("" : "+v"(dl[r4]));
      }
      s = kk == 0 ? s_first(fq, whole0, kv - k0 - 4 * hl, span) : mfma(fq, kf[kk], s);
      dp = mfma(fd, vf[kk], kk == 0 ? delta_init() : dp);
    }
    // the first step's dV/dK group: half -1 (stage 2, cleared)
#pragma unroll
    for (int f = 0; f < D; ++f) F[f] = read_frag(f, 1, 2, 0, 0);
    for (int it = 0; it < n_it3; it += 3) {
      item(it, Ci<0>{});
      item(it + 1, Ci<1>{});
      item(it + 2, Ci<2>{});
    }
    tail(Ci<2>{});
  }
  if (!kvv) return;
  bf16_t *base = (bf16_t *)a.dqkv + (int64_t)kv * ld;
#pragma unroll
  for (int i = 0; i < DT; ++i)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int d = 32 * i + 8 * r4 + 4 * hl;
      *(u32x2_t *)(base + (a.Hq + g) * HD + d) =
          u32x2_t{pack2(dk[i][4 * r4] * a.scale, dk[i][4 * r4 + 1] * a.scale),
                  pack2(dk[i][4 * r4 + 2] * a.scale, dk[i][4 * r4 + 3] * a.scale)};
      *(u32x2_t *)(base + (a.Hq + a.Hkv + g) * HD + d) =
          u32x2_t{pack2(dv[i][4 * r4], dv[i][4 * r4 + 1]), pack2(dv[i][4 * r4 + 2], dv[i][4 * r4 + 3])};
    }
}

__global__ __launch_bounds__(256) void attn_delta_bf16_kernel(AttnBwdArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (idx >= (int64_t)a.n_tok * a.Hq) return;
  const int row = (int)(idx / a.Hq), h = (int)(idx % a.Hq);
  const bf16_t *o = (const bf16_t *)a.o + (int64_t)row * a.Hq * a.hd + h * a.hd;
  const bf16_t *d = (const bf16_t *)a.dout + (int64_t)row * a.Hq * a.hd + h * a.hd;
  float s = 0.f;
  for (int c = lane; c < a.hd; c += 64) s += bf2f(o[c]) * bf2f(d[c]);
#pragma unroll
  for (int w = 32; w > 0; w >>= 1) s += __shfl_xor(s, w, 64);
  // stored negated: the dK/dV and dQ passes start their dP accumulators from
  // it, so that dP - delta costs no vector instruction
  if (lane == 0) a.delta[(int64_t)h * a.n_tok + row] = -s;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

bool attn_mfma_supported(int hd, const void *p0, const void *p1, const void *p2) {
  return (hd == 64 || hd == 128) && aligned16(p0) && aligned16(p1) && aligned16(p2);
}

// Waves per workgroup: every wave of a workgroup shares each staged K/V
// (forward, dQ) or Q/dO (dK/dV) tile.
constexpr int kFwdWaves = 8, kDqWaves = 8, kDkvWaves = 4;

int attn_fwd_mfma(const AttnArgs &a, hipStream_t s) {
  const int n_qt = (a.n_tok + 32 * kFwdWaves - 1) / (32 * kFwdWaves);
  const unsigned grid = (unsigned)n_qt * a.Hq;
  const int tk = timing_begin(s, AJ_KC_ATTN_FWD, 0.0);
  if (a.hd == 128) attn_fwd_mfma_kernel<128, kFwdWaves><<<grid, 64 * kFwdWaves, 0, s>>>(a, n_qt);
  else attn_fwd_mfma_kernel<64, kFwdWaves><<<grid, 64 * kFwdWaves, 0, s>>>(a, n_qt);
  timing_end(s, tk);
  return check_launch("attention forward (mfma)");
}

int attn_bwd_mfma(const AttnBwdArgs &a, hipStream_t s) {
  const int n_qt = (a.n_tok + 32 * kDqWaves - 1) / (32 * kDqWaves);
  const int n_kt = (a.n_tok + 32 * kDkvWaves - 1) / (32 * kDkvWaves);
  const int64_t nd = (int64_t)a.n_tok * a.Hq;
  const int tk = timing_begin(s, AJ_KC_ATTN_BWD, 0.0);
  attn_delta_bf16_kernel<<<(unsigned)((nd + 3) / 4), 256, 0, s>>>(a);
  if (a.hd == 128) {
    attn_dq_mfma_kernel<128, kDqWaves><<<(unsigned)n_qt * a.Hq, 64 * kDqWaves, 0, s>>>(a, n_qt);
    attn_dkv_mfma_kernel<128, kDkvWaves><<<(unsigned)n_kt * a.Hkv, 64 * kDkvWaves, 0, s>>>(a, n_kt);
  } else {
    attn_dq_mfma_kernel<64, kDqWaves><<<(unsigned)n_qt * a.Hq, 64 * kDqWaves, 0, s>>>(a, n_qt);
    attn_dkv_mfma_kernel<64, kDkvWaves><<<(unsigned)n_kt * a.Hkv, 64 * kDkvWaves, 0, s>>>(a, n_kt);
  }
  timing_end(s, tk);
  return check_launch("attention backward (mfma)");
}

}  // namespace aj
