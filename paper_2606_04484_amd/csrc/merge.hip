// Timeline merging on the GPU (Section 4.4.2, Algorithm 1), token-level Match
// and, further down, text-level Match (the Relaxed Matching Strategies).
//
// Algorithm 1 is a sequential double loop, but its result has a closed form
// that parallelises:
//   * Match leaves token ids unchanged, so whether T_j is a block-aligned
//     prefix of T_i (written T_j <= T_i) never changes while the loop runs;
//   * the largest i > j with T_j <= T_i is never absorbed itself (whatever
//     absorbed it would be a larger i with T_j <= i), and it is the first
//     candidate the descending loop offers j to, so
//         absorber(j) = max { i > j in j's episode : T_j <= T_i }   (or none);
//   * an absorbed timeline never absorbs (it is skipped when its turn comes),
//     so it hands over its ORIGINAL blocks; on a survivor's non-llm block k the
//     first transfer wins, and absorbed timelines arrive in descending j:
//         payload(s, k) = s's own block if llm, else the block k of the largest
//                         j absorbed into s whose block k is llm.
// Every token of a timeline is read by one pass that needs it: the prefix
// compare reads the tokens of every timeline that has a candidate absorber,
// the output pass the survivors'.  The compare splits each timeline into
// items of kCmpChunk tokens, so a long timeline is many short, evenly sized
// work items, and records each item's runs of llm tokens; the output pass
// takes a survivor's transferred log-probs from its absorbed timelines' runs
// (pulled, so nothing is cleared, voted into or read back per token).
// Kernels (token-level Match):
//   init_status     the call's status word and the scans' per-workgroup tallies
//   setup           offsets tile [0, n_tok) and [0, n_tl), every timeline starts
//                   a block; episode bounds per timeline; compare items per
//                   timeline
//   filter          one wavefront per timeline j: the first candidate, from the
//                   episode's last timeline down, that can hold T_j as a prefix
//                   (length, block boundary at |T_j|, first and last 64 tokens)
//   compare         one workgroup per kCmpChunk tokens of T_j: full compare with
//                   that candidate (a difference marks j), llm runs of the item
//   finalize        absorber = the candidate, or for a marked j the candidates
//                   below it compared in full (Algorithm 1's order); adds each
//                   wavefront's survivors and their tokens to the tally of the
//                   survivor-scan workgroup that holds them
//   resolve         one workgroup per kResSpan timelines, each starting from the
//                   tallies before it: survivor scan -> cu_seqlens, counts
//   emit            survivor tokens -> packed tok/pos/mask/old_logprob/adv (each
//                   workgroup a range of output positions); a survivor's non-llm
//                   token takes the log-prob of the largest absorbed timeline
//                   whose run covers its position; counts each range's targets
//                   and writes their bitmask; adds them to the tally of the
//                   offset-scan workgroup that holds the range
//   tgt_offsets     one workgroup per kTgtScanSpan ranges, each starting from
//                   the tallies before it: offsets of the per-range target
//                   counts
//   tgt_write       ascending masked targets from the bitmask, and each
//                   segment's first target (cu_targets)
#include <mutex>

#include "common.h"

// Workspace of aj_merge_timelines_noalloc: one copy per GPU, held for the
// life of the process.  Host code never passes this name to a kernel (on
// the host it is only a stand-in symbol); it uses the device address that
// hipGetSymbolAddress returns for the current device.
static constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kBlock = 256;
constexpr int kChunk = 1024;          // tokens per workgroup in the block-start compaction
constexpr int kCmpChunk = 2048;       // tokens per compare item: 32 rows of 64
constexpr int kRows = kCmpChunk / 64;                  // llm rows of 64 positions per item
constexpr int kRowsPerLane = (kRows + 63) / 64;        // rows per lane of a wavefront
constexpr int kCntBits = 14;          // item records hold positions (<= kCmpChunk) in 14 bits
constexpr int kRuns = 4;              // llm runs kept per compare item (more: marked kRuns + 1)
constexpr int kResPer = 8;            // timelines per thread of the survivor scan
constexpr int kResSpan = kResPer * 256;   // timelines per survivor-scan workgroup
constexpr int kTgtScanPer = 16;       // target chunks per thread of the target-offset scan
constexpr int kTgtScanSpan = kTgtScanPer * 256;   // target chunks per scan workgroup
static_assert(kCmpChunk % 1024 == 0 && kCmpChunk < (1 << kCntBits) &&
              (kRows <= 64 || kRows % 64 == 0), "item shape");
// Offsets that do not tile the input stop the merge (every count 0); bad flag
// bytes are reported and the token is treated as written (author 3: not llm).
constexpr int kFatal = AJ_DEVERR_OFFSETS | AJ_DEVERR_EMPTY | AJ_DEVERR_BLOCKS;

struct MergeArgs {
  int32_t n_traj, n_tl;
  int64_t n_tok;
  const int32_t *traj_tl_off;
  const int64_t *tl_tok_off;
  const int32_t *tok;
  const uint8_t *flags;
  const float *old_logprob, *adv;
  // outputs
  int32_t *absorber, *cu_seqlens, *seg_src, *cu_targets;
  int64_t *counts;
  int32_t *otok, *opos;
  uint8_t *omask;
  float *olp, *oadv;
  int32_t *targets;
  // workspace
  int32_t *status;      // [0] error bits seen by this call
  int32_t *tl_seg;      // [n_tl]
  int32_t *seg_base;    // [n_tl] first input token of each segment's survivor
  int32_t *range_rec;   // [n_ranges][kRecInts] per output range: first segment, transfer entries
  uint64_t *tbits;      // one bit per output position: a masked target
  int32_t *chunk_cnt;   // [n_chunks]
  int32_t *chunk_off;   // [n_chunks]
  int32_t *rblk;        // [n_rblk][4] per kResSpan timelines: survivors, their tokens, the
                        // longest (added up by the absorber pass), unused
  int32_t n_rblk;
  int32_t *tblk;        // [n_tblk] targets per kTgtScanSpan target chunks (added up by the
                        // passes that count each chunk's targets)
  int32_t n_tblk;
  int32_t *user_err;
  // token-level Match only.  Compare item (j, k) covers positions
  // [k * kCmpChunk, (k + 1) * kCmpChunk) of T_j and is slot
  // tl_tok_off[j] / kCmpChunk + j + k: the slots of consecutive timelines
  // never overlap, and n_tok / kCmpChunk + n_tl slots hold them all.
  int32_t n_slots;
  int32_t *ep_first;          // [n_tl] first timeline of the timeline's episode
  int32_t *ep_last;           // [n_tl] last timeline of the timeline's episode
  int32_t *cand;              // [n_tl] first candidate passing the filter, -1: none
  int32_t *miss;              // [n_tl] nonzero: the full compare with cand found a difference
  int4 *slot_rec;             // [n_slots] item: {j, first token of T_j, first token of the
                              // candidate (-1: no item), positions | k << kCntBits}
  int32_t *rcnt;              // [n_slots] llm runs of the item (kRuns + 1: more than kRuns)
  int32_t *runs;              // [n_slots][kRuns][2] [first, end) positions in the timeline
  // text-level Match only
  int32_t n_blk;
  const uint64_t *blk_text;   // [n_blk] text key per block
  int64_t *ti;                // [2] TI report, or null
  int32_t *blk_start;         // [n_blk+1] first token of each block, then n_tok
  int32_t *tl_blk;            // [n_tl+1]  first block of each timeline, then n_blk
  int32_t *blk_tl;            // [n_blk]   timeline of each block
  int32_t *blk_claim;         // [n_blk]   largest absorbed timeline with an llm block here
  int32_t *src_blk;           // [n_blk]   block whose tokens a survivor block carries (-1: none)
  int32_t *blk_off;           // [n_blk+1] output offset of each survivor block
  int32_t *dst_off;           // [n_blk]   output offset a source block lands at (-1: nowhere)
  int32_t *dst_pos;           // [n_blk]   its position inside the segment
};

AJ_DEV bool fatal(const MergeArgs &a) { return (a.status[0] & kFatal) != 0; }

AJ_DEV void raise(const MergeArgs &a, int bits) {
  atomicOr(a.status, bits);
  if (a.user_err) atomicOr(a.user_err, bits);
}

// Timeline handled by workgroup w of a one-per-timeline grid of n.  The
// hardware deals workgroups round-robin to the 8 XCDs, and episodes have
// equal turn counts, so w itself would put every episode's last timeline
// (its survivor) on one XCD; instead each XCD takes a contiguous eighth of
// the timelines (a bijection on [0, n)).
AJ_DEV int spread_timeline(int w, int n) {
  const int per = n / 8, rem = n % 8;
  const int x = w % 8;
  return x * per + (x < rem ? x : rem) + w / 8;
}

// Inclusive block scan of one int per thread; returns the inclusive value, *total
// gets the block sum.  blockDim.x must equal NT (a multiple of 64).
template <int NT>
AJ_DEV int block_scan_incl(int v, int *total) {
  __shared__ int wsum[NT / 64];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[wid] = x;
  __syncthreads();
  if (wid == 0) {
    int w = (lane < NT / 64) ? wsum[lane] : 0;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      int y = __shfl_up(w, o, 64);
      if (lane >= o) w += y;
    }
    if (lane < NT / 64) wsum[lane] = w;
  }
  __syncthreads();
  int res = x + (wid > 0 ? wsum[wid - 1] : 0);
  *total = wsum[NT / 64 - 1];
  __syncthreads();
  return res;
}

// Exclusive scan of the values v[r] (r < K) of one workgroup of NT threads,
// where thread (wave w, lane l) holds item w*64*K + r*64 + l: loads of
// consecutive items stay coalesced, the scan runs over the wave's items in
// order (64-lane scans with a carry), then over the waves.  v[r] becomes
// carry + the sum of the items before it; returns the total.
template <int NT, int K>
AJ_DEV int wave_items_scan(int (&v)[K], int carry) {
  __shared__ int wtot[NT / 64];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  int run = 0;
#pragma unroll
  for (int r = 0; r < K; ++r) {
    int x = v[r];
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    const int tot = __shfl(x, 63, 64);
    v[r] = run + x - v[r];
    run += tot;
  }
  if (lane == 0) wtot[wid] = run;
  __syncthreads();
  int before = carry, all = carry;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) {
    const int t = wtot[w];
    before += w < wid ? t : 0;
    all += t;
  }
#pragma unroll
  for (int r = 0; r < K; ++r) v[r] += before;
  __syncthreads();
  return all - carry;
}

AJ_DEV int validate_item(const MergeArgs &a, int t) {
  int bits = 0;
  if (t == 0) {
    if (a.traj_tl_off[0] != 0 || a.traj_tl_off[a.n_traj] != a.n_tl) bits |= AJ_DEVERR_OFFSETS;
    if (a.tl_tok_off[0] != 0 || a.tl_tok_off[a.n_tl] != a.n_tok) bits |= AJ_DEVERR_OFFSETS;
  }
  if (t < a.n_traj && a.traj_tl_off[t] > a.traj_tl_off[t + 1]) bits |= AJ_DEVERR_OFFSETS;
  if (t < a.n_tl) {
    const int64_t lo = a.tl_tok_off[t], hi = a.tl_tok_off[t + 1];
    if (lo < 0 || lo > hi || hi > a.n_tok) bits |= AJ_DEVERR_OFFSETS;
    else if (lo == hi) bits |= AJ_DEVERR_EMPTY;
    else if (!(a.flags[lo] & AJ_FLAG_BLOCK_START)) bits |= AJ_DEVERR_BAD_FLAGS;
  }
  return bits;
}

__global__ void init_status_kernel(MergeArgs a) {
  if (threadIdx.x < 4) a.status[threadIdx.x] = 0;
  if (a.ti && threadIdx.x < 2) a.ti[threadIdx.x] = 0;
  for (int i = threadIdx.x; i < 4 * a.n_rblk; i += blockDim.x) a.rblk[i] = 0;
  for (int i = threadIdx.x; i < a.n_tblk; i += blockDim.x) a.tblk[i] = 0;
}

// Adds one wavefront's survivors (surv: 0/1, len: the survivor's length) to
// the tally of the survivor-scan workgroup that holds timeline j (every lane's
// timeline lies in the same kResSpan-aligned range).  Integer sums and a
// maximum: the result does not depend on the order of the atomics.
AJ_DEV void tally_survivors(const MergeArgs &a, int j, int surv, int len) {
  int mx = len;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    surv += __shfl_xor(surv, o, 64);
    len += __shfl_xor(len, o, 64);
    mx = max(mx, __shfl_xor(mx, o, 64));
  }
  if ((threadIdx.x & 63) == 0 && surv > 0) {
    int32_t *t = a.rblk + 4 * (j / kResSpan);
    atomicAdd(t, surv);
    atomicAdd(t + 1, len);
    atomicMax(t + 2, mx);
  }
}

__global__ void validate_kernel(MergeArgs a) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  const int bits = validate_item(a, t);
  if (bits) raise(a, bits);
}

// The checks of validate, then the token merge's per-timeline tables:
// episode bounds and a cleared difference mark.  Tables are written only from
// offsets that are in range; if any are not, every later kernel stops.
__global__ __launch_bounds__(kBlock) void setup_kernel(MergeArgs a) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  const int bits = validate_item(a, t);
  if (bits) raise(a, bits);
  if (t < a.n_traj) {
    const int lo = a.traj_tl_off[t], hi = a.traj_tl_off[t + 1];
    if (0 <= lo && lo <= hi && hi <= a.n_tl)
      for (int i = lo; i < hi; ++i) {
        a.ep_first[i] = lo;
        a.ep_last[i] = hi - 1;
      }
  }
  if (t < a.n_tl) a.miss[t] = 0;
}

// One wavefront per timeline j: the first candidate i (from the episode's
// last timeline down, Algorithm 1's order) that passes the necessary
// conditions of T_j <= T_i on a few tokens: |T_i| >= |T_j|, a block starts in
// T_i right after T_j ends (or both end together), and the first and last 64
// positions of T_j agree in token id and block-start bit.  Candidates above
// the result fail a necessary condition, so they cannot absorb j.  Then the
// records of j's compare slots (and of the unused slots up to j + 1's first):
// everything a compare workgroup needs, in one load.
__global__ __launch_bounds__(kBlock) void filter_kernel(MergeArgs a) {
  const int j = blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (j >= a.n_tl) return;
  const bool bad = fatal(a);
  int c = -1;
  if (!bad) {
    const int last = a.ep_last[j];
    const int64_t bj = a.tl_tok_off[j], lj = a.tl_tok_off[j + 1] - bj;
    const int64_t q1 = min((int64_t)lane, lj - 1), q2 = max(lj - 1 - lane, (int64_t)0);
    const int32_t t0 = a.tok[bj], tj1 = a.tok[bj + q1], tj2 = a.tok[bj + q2];
    const int fj1 = a.flags[bj + q1] & AJ_FLAG_BLOCK_START;
    const int fj2 = a.flags[bj + q2] & AJ_FLAG_BLOCK_START;
    for (int ib = last; ib > j && c < 0; ib -= 64) {
      const int i = ib - lane;   // lane 0 holds the nearest the episode's end
      bool ok = false;
      int64_t bi = 0;
      if (i > j) {
        bi = a.tl_tok_off[i];
        const int64_t li = a.tl_tok_off[i + 1] - bi;
        ok = li >= lj && a.tok[bi] == t0 &&
             (li == lj || (a.flags[bi + lj] & AJ_FLAG_BLOCK_START) != 0);
      }
      uint64_t m = __ballot(ok);
      while (m) {
        const int l = __ffsll((unsigned long long)m) - 1;
        m &= m - 1;
        const int64_t b = __shfl(bi, l, 64);
        const bool eq = a.tok[b + q1] == tj1 && a.tok[b + q2] == tj2 &&
                        (a.flags[b + q1] & AJ_FLAG_BLOCK_START) == fj1 &&
                        (a.flags[b + q2] & AJ_FLAG_BLOCK_START) == fj2;
        if (__ballot(!eq) == 0) {
          c = ib - l;
          break;
        }
      }
    }
  }
  if (lane == 0) a.cand[j] = c;
  if (bad) return;
  const int64_t bj = a.tl_tok_off[j], ej = a.tl_tok_off[j + 1];
  const int64_t bc = c >= 0 ? a.tl_tok_off[c] : 0;
  // floor(b/C) + ceil((e-b)/C) <= floor(e/C) + 1: the slots of j end at or
  // before the first slot of j + 1
  const int s0 = (int)(bj / kCmpChunk) + j;
  const int s1 = (int)(ej / kCmpChunk) + j + 1;
  const int nk = (int)((ej - bj + kCmpChunk - 1) / kCmpChunk);
  for (int g = s0 + lane; g < s1; g += 64) {
    const int k = g - s0;
    int4 r = make_int4(-1, 0, -1, 0);
    if (k < nk && c >= 0) {
      const int p0 = k * kCmpChunk;
      r = make_int4(j, (int)(bj + p0), (int)(bc + p0),
                    (int)((uint32_t)min((int64_t)kCmpChunk, ej - bj - p0) | ((uint32_t)k << kCntBits)));
    }
    a.slot_rec[g] = r;
  }
}

// Compare rounds per item: each thread takes 4 consecutive positions a round.
constexpr int kCmpRounds = kCmpChunk / (4 * kBlock);
// Four token ids from a dword-aligned address (multi-dword global loads need
// only dword alignment).
typedef int32_t i32x4_a4 __attribute__((ext_vector_type(4), aligned(4)));

// Four consecutive flag bytes from any byte address, by aligned dword reads:
// the dword holding the first byte and, when that is not its first byte, the
// next one, which then holds the fourth (so neither read leaves the pages of
// the bytes asked for).
AJ_DEV uint32_t load_flags4(const uint8_t *p) {
  const uint32_t sh = (uint32_t)(reinterpret_cast<uintptr_t>(p) & 3);
  const uint32_t *w = reinterpret_cast<const uint32_t *>(p - sh);   // stays a global pointer
  const uint32_t lo = w[0];
  const uint32_t hi = sh ? w[1] : 0u;
  return __builtin_amdgcn_alignbyte(hi, lo, sh);
}

// One workgroup per compare slot: positions [p0, p0 + kCmpChunk) of T_j
// against the same positions of its candidate (token id and block-start
// bit); a difference marks j.  The llm tokens of the item, as rows of 64
// bits in LDS, become its runs [first, end), kRuns at most (more: the item is
// marked and the output pass reads its flags instead).  Each thread takes 4
// consecutive positions a round: 16-byte token loads and 4 flag bytes per
// dword.  Slots are dealt to the XCDs in contiguous ranges, so the items of
// one episode -- which read the same candidate -- share an L2.
__global__ __launch_bounds__(kBlock) void compare_kernel(MergeArgs a) {
  const int g = spread_timeline(blockIdx.x, a.n_slots);
  const int4 rc = a.slot_rec[g];
  if (fatal(a) || rc.z < 0) return;
  // the record is the workgroup's: its fields live in scalar registers
  const int j = __builtin_amdgcn_readfirstlane(rc.x);
  const int32_t uj = __builtin_amdgcn_readfirstlane(rc.y);   // first token of the item in T_j
  const int32_t uc = __builtin_amdgcn_readfirstlane(rc.z);   // ... and in the candidate
  const uint32_t w = (uint32_t)__builtin_amdgcn_readfirstlane(rc.w);
  const int n = (int)(w & ((1u << kCntBits) - 1));          // positions, 1..kCmpChunk
  const int p0 = (int)(w >> kCntBits) * kCmpChunk;
  const int32_t *tj0 = a.tok + uj, *tc0 = a.tok + uc;
  const uint8_t *fj0 = a.flags + uj, *fc0 = a.flags + uc;
  __shared__ uint64_t rows[kCmpChunk / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  i32x4_a4 tj[kCmpRounds], tc[kCmpRounds];
  uint32_t fj[kCmpRounds], fc[kCmpRounds];
#pragma unroll
  for (int r = 0; r < kCmpRounds; ++r) {
    const int q = r * 4 * kBlock + 4 * (int)threadIdx.x;
    if (q + 4 <= n) {
      tj[r] = *reinterpret_cast<const i32x4_a4 *>(tj0 + (uint32_t)q);
      tc[r] = *reinterpret_cast<const i32x4_a4 *>(tc0 + (uint32_t)q);
      fj[r] = load_flags4(fj0 + (uint32_t)q);
      fc[r] = load_flags4(fc0 + (uint32_t)q);
    } else {   // the item's ragged end: clamped single reads
      uint32_t xj = 0, xc = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t qq = (uint32_t)min(q + e, n - 1);
        tj[r][e] = tj0[qq];
        tc[r][e] = tc0[qq];
        xj |= (uint32_t)fj0[qq] << (8 * e);
        xc |= (uint32_t)fc0[qq] << (8 * e);
      }
      fj[r] = xj;
      fc[r] = xc;
    }
  }
  int diff = 0, bad = 0;
#pragma unroll
  for (int r = 0; r < kCmpRounds; ++r) {
    const int q = r * 4 * kBlock + 4 * (int)threadIdx.x;
    const int n_in = max(0, min(4, n - q));                     // positions of the group in the item
    const uint32_t in = n_in == 4 ? 0xffffffffu : (1u << (8 * n_in)) - 1u;
#pragma unroll
    for (int e = 0; e < 4; ++e) diff |= e < n_in && tj[r][e] != tc[r][e];
    diff |= ((fj[r] ^ fc[r]) & in & 0x04040404u) != 0;
    bad |= (fj[r] & (fj[r] >> 1) & in & 0x01010101u) != 0;     // author 3
    const uint32_t llm = (fj[r] >> 1) & ~fj[r] & in & 0x01010101u;   // author 2
    const uint32_t n4 = (llm & 1u) | ((llm >> 7) & 2u) | ((llm >> 14) & 4u) | ((llm >> 21) & 8u);
    // the wave's 256 positions are 4 rows of 64, 16 lanes x 4 positions each:
    // a row is its 16 lanes' nibbles side by side (an OR over the group)
    uint64_t row = (uint64_t)n4 << (4 * (lane & 15));
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) row |= __shfl_xor(row, o, 64);
    if ((lane & 15) == 0) rows[r * (kBlock / 16) + wave * 4 + (lane >> 4)] = row;   // bit = position % 64
  }
  if (bad) raise(a, AJ_DEVERR_BAD_FLAGS);
  if (__syncthreads_or(diff) && threadIdx.x == 0) atomicOr(a.miss + j, 1);
  if (wave != 0) return;
  // runs: a start is an llm position whose predecessor in the item is not,
  // an end one whose successor is not; the k-th start pairs with the k-th end
  // lane l holds rows kRowsPerLane * l ... (positions 64 * row + bit)
  constexpr int RL = kRowsPerLane;
  const int nl = kRows / RL;   // lanes holding rows
  uint64_t m[RL], st[RL], en[RL];
#pragma unroll
  for (int i = 0; i < RL; ++i) m[i] = lane < nl ? rows[RL * lane + i] : 0;
  const uint64_t before = lane > 0 && lane < nl ? rows[RL * lane - 1] >> 63 : 0;
  const uint64_t after = lane < nl - 1 ? rows[RL * (lane + 1)] & 1 : 0;
  int xs = 0, xe = 0;
#pragma unroll
  for (int i = 0; i < RL; ++i) {
    const uint64_t prev = i == 0 ? before : m[i - 1] >> 63;
    const uint64_t next = i == RL - 1 ? after : m[i + 1] & 1;
    st[i] = m[i] & ~((m[i] << 1) | prev);
    en[i] = m[i] & ~((m[i] >> 1) | (next << 63));
    xs += __popcll(st[i]);
    xe += __popcll(en[i]);
  }
  const int ns = xs, ne = xe;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int ys = __shfl_up(xs, o, 64), ye = __shfl_up(xe, o, 64);
    if (lane >= o) { xs += ys; xe += ye; }
  }
  const int total = __shfl(xs, 63, 64);
  int32_t *dst = a.runs + (int64_t)g * (2 * kRuns);
  int rs = xs - ns, re = xe - ne;
#pragma unroll
  for (int i = 0; i < RL; ++i) {
    const int base = p0 + 64 * (RL * lane + i);
    for (; st[i] && rs < kRuns; ++rs, st[i] &= st[i] - 1)
      dst[2 * rs] = base + __ffsll((unsigned long long)st[i]) - 1;
    for (; en[i] && re < kRuns; ++re, en[i] &= en[i] - 1)
      dst[2 * re + 1] = base + __ffsll((unsigned long long)en[i]);
  }
  if (lane == 0) a.rcnt[g] = total > kRuns ? kRuns + 1 : total;
}

// Algorithm 1's answer for j from the candidates i = from, from - 1, ..., j + 1
// (every candidate above `from` is known not to hold T_j as a prefix): the
// first whose block-aligned prefix equals T_j, compared in full by the whole
// workgroup with early exit; -1 if none.
AJ_DEV int search_absorber(const MergeArgs &a, int j, int from) {
  const int64_t bj = a.tl_tok_off[j];
  const int64_t lj = a.tl_tok_off[j + 1] - bj;
  for (int i = from; i > j; --i) {
    const int64_t bi = a.tl_tok_off[i];
    const int64_t li = a.tl_tok_off[i + 1] - bi;
    if (li < lj) continue;
    // block-aligned: T_i must start a new block right where T_j ends
    if (li > lj && !(a.flags[bi + lj] & AJ_FLAG_BLOCK_START)) continue;
    bool equal = true;
    for (int64_t base = 0; base < lj; base += 8 * kBlock) {
      int bad = 0;
      int32_t tj[8], ti[8];
      uint8_t fj[8], fi[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) {   // clamped (lj >= 1): all loads issued together
        const int64_t p = min(base + r * kBlock + (int64_t)threadIdx.x, lj - 1);
        tj[r] = a.tok[bj + p]; ti[r] = a.tok[bi + p];
        fj[r] = a.flags[bj + p]; fi[r] = a.flags[bi + p];
      }
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        bad |= tj[r] != ti[r];
        bad |= ((fj[r] ^ fi[r]) & AJ_FLAG_BLOCK_START) != 0;
      }
      if (__syncthreads_or(bad)) { equal = false; break; }
    }
    if (equal) return i;
  }
  return -1;
}

// Timelines per finalize workgroup.
constexpr int kFinPer = 64;

// absorber[j] = the candidate when the full compare found no difference;
// for a marked j the workgroup searches the candidates below it (the rare
// case: a prefix that agrees at both ends and differs inside).
__global__ __launch_bounds__(kBlock) void finalize_kernel(MergeArgs a) {
  static_assert(kFinPer == 64 && kResSpan % kFinPer == 0, "one wavefront of timelines");
  __shared__ int todo[kFinPer], found[kFinPer];
  __shared__ int n_todo;
  if (threadIdx.x == 0) n_todo = 0;
  __syncthreads();
  const bool bad = fatal(a);
  const int j = blockIdx.x * kFinPer + (int)threadIdx.x;
  int ab = -1, slot = -1;
  if (threadIdx.x < kFinPer && j < a.n_tl) {
    ab = bad ? -1 : a.cand[j];
    if (ab >= 0 && a.miss[j] != 0) todo[slot = atomicAdd(&n_todo, 1)] = j;
    else a.absorber[j] = ab;
  }
  __syncthreads();
  const int n = n_todo;
  for (int f = 0; f < n; ++f) {
    const int jj = todo[f];
    const int r = search_absorber(a, jj, a.cand[jj] - 1);
    if (threadIdx.x == 0) {
      a.absorber[jj] = r;
      found[f] = r;
    }
  }
  __syncthreads();
  // the survivors among the workgroup's timelines, for the survivor scan
  if (threadIdx.x < kFinPer && !bad) {
    if (slot >= 0) ab = found[slot];
    const bool surv = j < a.n_tl && ab < 0;
    tally_survivors(a, j, surv ? 1 : 0, surv ? (int)(a.tl_tok_off[j + 1] - a.tl_tok_off[j]) : 0);
  }
}

// No merge: every timeline survives.
__global__ __launch_bounds__(kBlock) void fill_absorber_kernel(MergeArgs a) {
  const int t = blockIdx.x * kBlock + threadIdx.x;
  const bool surv = t < a.n_tl && !fatal(a);
  if (t < a.n_tl) a.absorber[t] = -1;
  tally_survivors(a, t, surv ? 1 : 0, surv ? (int)(a.tl_tok_off[t + 1] - a.tl_tok_off[t]) : 0);
}

// The survivors' scan, one workgroup per kResSpan timelines: wave w of
// workgroup b holds the kResPer * 64 consecutive timelines from
// b * kResSpan + w * 64 * kResPer (lane l every 64th), so the loads stay
// coalesced.  A workgroup's offsets start from the tallies of the workgroups
// before it (written by the absorber pass); the last one writes the totals.
__global__ __launch_bounds__(kBlock) void resolve_kernel(MergeArgs a) {
  static_assert(kResSpan == kResPer * kBlock, "timelines per workgroup");
  __shared__ int red[3][kBlock / 64];
  const bool bad = fatal(a);
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int b = blockIdx.x;
  const bool last = b == (int)gridDim.x - 1;
  // survivors and tokens before this workgroup's timelines; the longest
  // survivor of all (the last workgroup only)
  int ps = 0, pt = 0, pm = 0;
  for (int i = threadIdx.x; i < (last ? a.n_rblk : b); i += kBlock) {
    if (i < b) {
      ps += a.rblk[4 * i];
      pt += a.rblk[4 * i + 1];
    }
    pm = max(pm, a.rblk[4 * i + 2]);
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    ps += __shfl_xor(ps, o, 64);
    pt += __shfl_xor(pt, o, 64);
    pm = max(pm, __shfl_xor(pm, o, 64));
  }
  if (lane == 0) {
    red[0][wid] = ps;
    red[1][wid] = pt;
    red[2][wid] = pm;
  }
  __syncthreads();
  ps = pt = pm = 0;
#pragma unroll
  for (int w = 0; w < kBlock / 64; ++w) {
    ps += red[0][w];
    pt += red[1][w];
    pm = max(pm, red[2][w]);
  }
  if (bad) ps = pt = pm = 0;
  const int i0 = b * kResSpan + wid * 64 * kResPer + lane;
  int seg[kResPer], tok[kResPer];
#pragma unroll
  for (int r = 0; r < kResPer; ++r) {
    seg[r] = tok[r] = 0;
    if (a.n_tl > 0) {   // clamped, not guarded: the loads issue together
      const int i = min(i0 + 64 * r, a.n_tl - 1);
      const bool ok = !bad && i0 + 64 * r < a.n_tl;
      const int ab = a.absorber[i];
      const int l = (int)(a.tl_tok_off[i + 1] - a.tl_tok_off[i]);
      seg[r] = ok && ab < 0;
      tok[r] = seg[r] ? l : 0;
    }
  }
  uint32_t surv = 0;
#pragma unroll
  for (int r = 0; r < kResPer; ++r) surv |= (uint32_t)seg[r] << r;
  const int tot_s = wave_items_scan<kBlock, kResPer>(seg, ps);
  const int tot_l = wave_items_scan<kBlock, kResPer>(tok, pt);
#pragma unroll
  for (int r = 0; r < kResPer; ++r) {
    const int i = i0 + 64 * r;
    if (i >= a.n_tl) continue;
    if ((surv >> r) & 1) {
      a.tl_seg[i] = seg[r];
      a.seg_src[seg[r]] = i;
      a.seg_base[seg[r]] = (int32_t)a.tl_tok_off[i];
      a.cu_seqlens[seg[r]] = tok[r];
    } else {
      a.tl_seg[i] = -1;
    }
  }
  if (last && threadIdx.x == 0) {
    a.cu_seqlens[ps + tot_s] = pt + tot_l;
    a.counts[0] = ps + tot_s;
    a.counts[1] = pt + tot_l;
    a.counts[2] = 0;
    a.counts[3] = pm;
  }
}

// Largest s in [lo, hi] with cu[s] <= o (cu ascending, cu[lo] <= o), by one
// wave: 64 probes a step, so a few dependent reads for any segment count.
AJ_DEV int wave_search(const int32_t *cu, int64_t o, int lo, int hi) {
  const int lane = threadIdx.x & 63;
  while (lo < hi) {
    const int64_t span = (int64_t)hi - lo + 1;
    const int q = lo + (int)(span * lane / 64);
    // q ascends with the lane and lane 0 probes lo, so the lanes with
    // cu[q] <= o are a non-empty prefix
    const uint64_t m = __ballot(cu[q] <= o);
    const int l = 63 - __clzll(m);
    const int nlo = __shfl(q, l, 64);
    const int nhi = l < 63 ? __shfl(q, l + 1, 64) - 1 : hi;
    lo = nlo;
    hi = nhi;
  }
  return lo;
}

// Largest s in [lo, hi] with cu[s] <= o, one thread.
AJ_DEV int thread_search(const int32_t *cu, int64_t o, int lo, int hi) {
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu[mid] <= o) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Output positions [ob, ob + kEmitSpan) per range.  A first pass (range,
// one wavefront per range) finds the range's first segment and, for token
// Match, its transfer entries; the output pass (emit) then needs one record
// load before its bulk reads.  Transfers: the candidates j of a segment's
// survivor s are the earlier timelines of its episode with absorber[j] == s;
// their llm runs that fall inside the range become entries [lo, hi) of output
// positions with the distance to the source token.  A non-llm survivor token
// takes the largest source among the entries that cover it (source token
// indices grow with the timeline index, so that is the largest absorbed j,
// the transfer Algorithm 1 keeps).
constexpr int kEmitPer = 8;
constexpr int kEmitSpan = kEmitPer * kBlock;
constexpr int kEmitWgs = 2048;   // grid of the stride loops when the occupancy query fails
constexpr int kRangeEnt = 8;     // transfer entries per range record (more: every output walks)
constexpr int kRecInts = 32;     // {first segment, entries or -1 (walk), kRangeEnt x {lo, hi, dl}}
static_assert(2 + 3 * kRangeEnt <= kRecInts && kRecInts <= 64, "one record per wavefront load");
static_assert(kEmitSpan <= kCmpChunk, "a range meets at most two compare items of a timeline");

// Source token of position p of survivor s (whose own token there is not
// llm): the token at p of the largest j absorbed into s whose token there is
// llm, or -1.  One thread, candidates from the nearest down; used for ranges
// a record cannot describe (more than 64 segments or kRangeEnt entries).
AJ_DEV int64_t claim_walk(const MergeArgs &a, int s, int p) {
  for (int j = s - 1; j >= a.ep_first[s]; --j) {
    if (a.absorber[j] != s) continue;
    const int64_t bj = a.tl_tok_off[j];
    if (p >= a.tl_tok_off[j + 1] - bj) continue;
    const int g = (int)(bj / kCmpChunk) + j + p / kCmpChunk;
    const int n = a.rcnt[g];
    bool hit = false;
    if (n > kRuns) {
      hit = (a.flags[bj + p] & AJ_AUTHOR_MASK) == AJ_AUTHOR_LLM;
    } else {
      const int32_t *rr = a.runs + (int64_t)g * (2 * kRuns);
      for (int r = 0; r < n; ++r) hit |= p >= rr[2 * r] && p < rr[2 * r + 1];
    }
    if (hit) return bj + p;
  }
  return -1;
}

// One wavefront per output range: the first segment (64 probes a step) and,
// with use_claims, the transfer entries of the range's segments -- lanes
// take (segment, candidate) pairs, each pair's runs in the range's positions
// become entries (an item whose runs overflowed gives one entry whose flag
// bytes are checked per output).
__global__ __launch_bounds__(kBlock) void range_kernel(MergeArgs a, int use_claims) {
  __shared__ int n_ent[kBlock / 64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = blockIdx.x * (kBlock / 64) + wave;
  if (fatal(a)) return;
  const int64_t n_out = a.counts[1];
  const int n_seg = (int)a.counts[0];
  const int64_t ob = (int64_t)r * kEmitSpan;
  if (ob >= n_out) return;
  const int64_t oe = min(ob + kEmitSpan, n_out);
  const int s0 = wave_search(a.cu_seqlens, ob, 0, n_seg - 1);
  int32_t *rec = a.range_rec + (int64_t)r * kRecInts;
  int ne = 0;
  if (use_claims) {
    if (lane == 0) n_ent[wave] = 0;
    const int sl = s0 + lane;
    const int cs = a.cu_seqlens[min(sl, n_seg)];
    const int c64 = a.cu_seqlens[min(s0 + 64, n_seg)];
    const bool in = sl < n_seg && cs < oe;
    const int sv = in ? a.seg_src[sl] : 0;
    const int ce = in ? a.cu_seqlens[sl + 1] : 0;
    const int np = in ? sv - a.ep_first[sv] : 0;
    int excl = np;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(excl, o, 64);
      if (lane >= o) excl += y;
    }
    const int total = __shfl(excl, 63, 64);
    excl -= np;
    if (s0 + 64 < n_seg && c64 < oe) ne = -1;   // more than 64 segments: walk
    for (int pb = 0; pb < total && ne >= 0; pb += 64) {
      const int idx = pb + lane;
      int k = 0;   // the lane whose pair range holds idx
#pragma unroll
      for (int st = 32; st > 0; st >>= 1) {
        const int v = __shfl(excl, min(k + st, 63), 64);
        if (k + st < 64 && v <= idx) k += st;
      }
      const int svk = __shfl(sv, k, 64), csk = __shfl(cs, k, 64), cek = __shfl(ce, k, 64);
      const int j = svk - 1 - (idx - __shfl(excl, k, 64));
      if (idx < total && a.absorber[j] == svk) {
        const int64_t bj = a.tl_tok_off[j];
        const int lj = (int)(a.tl_tok_off[j + 1] - bj);
        const int q0 = (int)(max(ob, (int64_t)csk) - csk);
        const int q1 = (int)min(min(oe, (int64_t)cek) - csk, (int64_t)lj);
        const int dl = (int)(bj - csk);   // source token = output position + dl
        for (int kk = q0 / kCmpChunk; kk * kCmpChunk < q1; ++kk) {
          const int g = (int)(bj / kCmpChunk) + j + kk;
          const int nr = a.rcnt[g];
          const int32_t *rr = a.runs + (int64_t)g * (2 * kRuns);
          for (int x = 0; x < (nr > kRuns ? 1 : nr); ++x) {
            int lo, hi;
            uint32_t ovf = 0;
            if (nr > kRuns) {
              lo = max(q0, kk * kCmpChunk);
              hi = min(q1, (kk + 1) * kCmpChunk);
              ovf = 0x80000000u;
            } else {
              lo = max(rr[2 * x], q0);
              hi = min(rr[2 * x + 1], q1);
            }
            if (lo >= hi) continue;
            const int e = atomicAdd(&n_ent[wave], 1);
            if (e < kRangeEnt) {
              rec[2 + 3 * e] = csk + lo;
              rec[3 + 3 * e] = (int32_t)((uint32_t)(csk + hi) | ovf);
              rec[4 + 3 * e] = dl;
            }
          }
        }
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
      ne = n_ent[wave];
      if (ne > kRangeEnt) ne = -1;
    }
  }
  if (lane == 0) {
    rec[0] = s0;
    rec[1] = ne;
  }
}

// One output of a range the record cannot describe (more than 64 segments
// or kRangeEnt transfer entries): its segment by search, its transfer by
// walking the candidates.  Writes the output; returns 1 for a target, 0 for
// a masked token without one, -1 for an unmasked token.
AJ_DEV int emit_one(const MergeArgs &a, int32_t o, int n_seg, int use_claims, int *bad) {
  const int sg = thread_search(a.cu_seqlens, o, 0, n_seg - 1);
  const int32_t pos = o - a.cu_seqlens[sg];
  const int32_t u = a.seg_base[sg] + pos;
  const uint8_t f = a.flags[u];
  int64_t src = (f & AJ_AUTHOR_MASK) == AJ_AUTHOR_LLM ? (int64_t)u : -1;
  if (src < 0 && use_claims) src = claim_walk(a, a.seg_src[sg], pos);
  *bad |= (f & AJ_AUTHOR_MASK) == AJ_AUTHOR_MASK;
  a.otok[o] = a.tok[u];
  a.opos[o] = pos;
  a.omask[o] = src >= 0;
  a.olp[o] = src >= 0 ? a.old_logprob[src] : 0.f;
  a.oadv[o] = src >= 0 ? a.adv[src] : 0.f;
  return src < 0 ? -1 : (pos != 0 ? 1 : 0);
}

__global__ __launch_bounds__(kBlock) void emit_kernel(MergeArgs a, int use_claims) {
  if (fatal(a)) return;
  const int64_t n_out = a.counts[1];
  const int n_seg = (int)a.counts[0];
  __shared__ int32_t seg_cu[65];
  __shared__ int32_t seg_base[64];
  __shared__ int n_ent;
  __shared__ int32_t ent[3 * kRangeEnt];   // {lo, hi | overflow << 31, dl}
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int bad = 0;
  for (int64_t ob = (int64_t)blockIdx.x * kEmitSpan; ob < n_out;
       ob += (int64_t)gridDim.x * kEmitSpan) {
    const int64_t oe = min(ob + kEmitSpan, n_out);
    if (threadIdx.x < 64) {
      const int32_t *rec = a.range_rec + ob / kEmitSpan * kRecInts;
      const int v = lane < kRecInts ? rec[lane] : 0;
      const int s0 = __shfl(v, 0, 64), ne = __shfl(v, 1, 64);
      if (lane >= 2 && lane < 2 + 3 * kRangeEnt) ent[lane - 2] = v;
      const int sl = s0 + lane;
      seg_cu[lane] = a.cu_seqlens[min(sl, n_seg)];            // cu[n_seg] = n_out
      if (lane == 0) seg_cu[64] = s0 + 64 <= n_seg ? a.cu_seqlens[s0 + 64] : INT32_MAX;
      seg_base[lane] = sl < n_seg ? a.seg_base[sl] : 0;
      if (lane == 0) n_ent = use_claims ? ne : 0;
    }
    __syncthreads();
    const int ne = n_ent;
    int n_tgt = 0;
    if (ne >= 0 && seg_cu[64] >= oe) {
      // every output in a table segment, transfers as entries: token indices
      // and output positions fit in 32 bits (n_tok < 2^31)
      int32_t u[kEmitPer], pos[kEmitPer];
#pragma unroll
      for (int r = 0; r < kEmitPer; ++r) {
        const int32_t o = (int32_t)min(ob + r * kBlock + (int64_t)threadIdx.x, n_out - 1);
        int k = 0;   // largest k with seg_cu[k] <= o, in LDS
#pragma unroll
        for (int st = 32; st > 0; st >>= 1)
          if (k + st < 64 && seg_cu[k + st] <= o) k += st;
        pos[r] = o - seg_cu[k];
        u[r] = seg_base[k] + pos[r];
      }
      uint8_t f[kEmitPer];
      int32_t t[kEmitPer];
#pragma unroll
      for (int r = 0; r < kEmitPer; ++r) {   // issued together
        f[r] = a.flags[u[r]];
        t[r] = a.tok[u[r]];
      }
      int32_t src[kEmitPer];
#pragma unroll
      for (int r = 0; r < kEmitPer; ++r) {
        const int32_t o = (int32_t)(ob + r * kBlock + threadIdx.x);
        src[r] = -1;
        if ((f[r] & AJ_AUTHOR_MASK) == AJ_AUTHOR_LLM) {   // the survivor's own llm token
          src[r] = u[r];
          continue;
        }
        for (int e = 0; e < ne; ++e) {
          const uint32_t hi = (uint32_t)ent[3 * e + 1];
          if (o < ent[3 * e] || (uint32_t)o >= (hi & 0x7fffffffu)) continue;
          const int32_t s = o + ent[3 * e + 2];
          if ((hi >> 31) && (a.flags[s] & AJ_AUTHOR_MASK) != AJ_AUTHOR_LLM) continue;
          src[r] = max(src[r], s);
        }
      }
      float lp[kEmitPer], ad[kEmitPer];
#pragma unroll
      for (int r = 0; r < kEmitPer; ++r) {   // only tokens that carry a log-prob
        lp[r] = 0.f;
        ad[r] = 0.f;
        if (src[r] >= 0) {
          lp[r] = a.old_logprob[src[r]];
          ad[r] = a.adv[src[r]];
        }
      }
#pragma unroll
      for (int r = 0; r < kEmitPer; ++r) {
        const int64_t o = ob + r * kBlock + threadIdx.x;
        const bool in = o < n_out;
        const bool has = in && src[r] >= 0;
        const bool tgt = has && pos[r] != 0;
        const uint64_t word = __ballot(tgt);
        if (lane == 0) a.tbits[ob / 64 + r * (kBlock / 64) + wave] = word;
        if (!in) continue;
        bad |= (f[r] & AJ_AUTHOR_MASK) == AJ_AUTHOR_MASK;
        a.otok[o] = t[r];
        a.opos[o] = pos[r];
        a.omask[o] = has;
        a.olp[o] = lp[r];
        a.oadv[o] = ad[r];
        n_tgt += tgt;
      }
    } else {
#pragma unroll 1
      for (int r = 0; r < kEmitPer; ++r) {
        const int64_t o = ob + r * kBlock + threadIdx.x;
        const int res = o < n_out ? emit_one(a, (int32_t)o, n_seg, use_claims, &bad) : -1;
        const uint64_t word = __ballot(res > 0);
        if (lane == 0) a.tbits[ob / 64 + r * (kBlock / 64) + wave] = word;
        n_tgt += res > 0;
      }
    }
    // the span's target count for the compaction (chunk = span)
    int tot;
    block_scan_incl<kBlock>(n_tgt, &tot);
    if (threadIdx.x == 0) {
      a.chunk_cnt[ob / kEmitSpan] = tot;
      if (tot) atomicAdd(&a.tblk[ob / kEmitSpan / kTgtScanSpan], tot);
    }
  }
  if (bad) raise(a, AJ_DEVERR_BAD_FLAGS);
}

// Target flags of the kTgtPer outputs from o0 (bit r: output o0 + r is a
// masked token that is not a segment's first); all loads issued together,
// vector ones when the outputs are aligned.  kTgtChunk equals emit's span,
// so emit can count a chunk's targets as it writes them.
constexpr int kTgtPer = 8;
constexpr int kTgtChunk = kTgtPer * kBlock;   // outputs per workgroup
static_assert(kTgtChunk == kEmitSpan, "emit counts the target chunks");

AJ_DEV uint32_t target_bits(const MergeArgs &a, int64_t o0, int64_t n_out) {
  uint32_t bits = 0;
  if (o0 + kTgtPer <= n_out && ((uintptr_t)a.omask & 7) == 0 && ((uintptr_t)a.opos & 15) == 0) {
    const uint2 m = *reinterpret_cast<const uint2 *>(a.omask + o0);
    const int4 q0 = *reinterpret_cast<const int4 *>(a.opos + o0);
    const int4 q1 = *reinterpret_cast<const int4 *>(a.opos + o0 + 4);
    const int pv[8] = {q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w};
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const uint32_t mb = ((r < 4 ? m.x : m.y) >> (8 * (r & 3))) & 0xff;
      bits |= (uint32_t)(mb != 0 && pv[r] != 0) << r;
    }
  } else {
#pragma unroll
    for (int r = 0; r < kTgtPer; ++r) {
      const int64_t o = o0 + r;
      if (o < n_out && a.omask[o] && a.opos[o] != 0) bits |= 1u << r;
    }
  }
  return bits;
}

// The text path's target count per chunk (token-level emit counts its own),
// with the chunk's target bitmask.
__global__ __launch_bounds__(kBlock) void tgt_count_kernel(MergeArgs a) {
  const int64_t n_out = fatal(a) ? 0 : a.counts[1];
  const int64_t o0 = (int64_t)blockIdx.x * kTgtChunk + threadIdx.x * kTgtPer;
  const uint32_t bits = target_bits(a, o0, n_out);
  // 8 bits per thread: thread t holds byte t % 8 of the chunk's word t / 8
  const int lane = threadIdx.x & 63;
  uint64_t w = (uint64_t)bits << (8 * (lane & 7));
#pragma unroll
  for (int o = 1; o < 8; o <<= 1) w |= __shfl_xor(w, o, 64);
  if ((lane & 7) == 0) a.tbits[o0 / 64] = w;
  const int c = __popc(bits);
  int tot;
  block_scan_incl<kBlock>(c, &tot);
  if (threadIdx.x == 0) {
    a.chunk_cnt[blockIdx.x] = tot;
    if (tot) atomicAdd(&a.tblk[blockIdx.x / kTgtScanSpan], tot);
  }
}

// Exclusive offsets of the per-chunk target counts, one workgroup per
// kTgtScanSpan chunks, starting from the tallies of the chunks before it; the
// workgroup holding the last chunk with outputs (or workgroup 0, when there
// are none) writes the total to counts[2].
__global__ __launch_bounds__(kBlock) void tgt_offsets_kernel(MergeArgs a) {
  static_assert(kTgtScanSpan == kTgtScanPer * kBlock, "chunks per workgroup");
  __shared__ int red[kBlock / 64];
  const int n_used = (int)((a.counts[1] + kTgtChunk - 1) / kTgtChunk);
  const int b = blockIdx.x;
  if (b > 0 && b * kTgtScanSpan >= n_used) return;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  int p = 0;
  for (int i = threadIdx.x; i < b; i += kBlock) p += a.tblk[i];
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) p += __shfl_xor(p, o, 64);
  if (lane == 0) red[wid] = p;
  __syncthreads();
  p = 0;
#pragma unroll
  for (int w = 0; w < kBlock / 64; ++w) p += red[w];
  const int c0 = b * kTgtScanSpan + wid * 64 * kTgtScanPer + lane;
  int v[kTgtScanPer];
#pragma unroll
  for (int r = 0; r < kTgtScanPer; ++r) v[r] = c0 + 64 * r < n_used ? a.chunk_cnt[c0 + 64 * r] : 0;
  const int tot = wave_items_scan<kBlock, kTgtScanPer>(v, p);
#pragma unroll
  for (int r = 0; r < kTgtScanPer; ++r)
    if (c0 + 64 * r < n_used) a.chunk_off[c0 + 64 * r] = v[r];
  if (threadIdx.x == 0 && b == (n_used > 0 ? (n_used - 1) / kTgtScanSpan : 0)) a.counts[2] = p + tot;
}

// Exclusive offsets of the per-chunk counts by one workgroup, 1024 * kScanPer
// chunks a round: the block-start compaction, whose total must equal n_blk.
constexpr int kScanPer = 16;

__global__ __launch_bounds__(1024) void blk_scan_kernel(MergeArgs a, int n_chunks) {
  const int n_used = n_chunks;
  int carry = 0;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  for (int base = 0; base < n_used; base += 1024 * kScanPer) {
    const int c0 = base + wid * 64 * kScanPer + lane;
    int v[kScanPer];
#pragma unroll
    for (int r = 0; r < kScanPer; ++r) v[r] = c0 + 64 * r < n_used ? a.chunk_cnt[c0 + 64 * r] : 0;
    carry += wave_items_scan<1024, kScanPer>(v, carry);
#pragma unroll
    for (int r = 0; r < kScanPer; ++r)
      if (c0 + 64 * r < n_used) a.chunk_off[c0 + 64 * r] = v[r];
  }
  if (threadIdx.x == 0 && !fatal(a) && carry != a.n_blk) raise(a, AJ_DEVERR_BLOCKS);
}

// A grid-stride walk over the chunks that hold outputs (the merged length is
// known only on the device), one wavefront per chunk: lane l takes outputs
// [32 l, 32 l + 32) (half a bitmask word), a wavefront scan of the lanes'
// target counts places them in the wavefront's LDS row, which is then stored
// contiguously; one round trip of loads per chunk, no wavefront waits on
// another.  Then a walk over the segments: cu_targets[s] = the number of
// targets before the segment's first output.
AJ_DEV void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

__global__ __launch_bounds__(kBlock) void tgt_write_kernel(MergeArgs a) {
  static_assert(kTgtChunk == 64 * 32, "32 outputs per lane of a wavefront");
  __shared__ int32_t row[kBlock / 64][kTgtChunk];
  const int64_t n_out = fatal(a) ? 0 : a.counts[1];
  const int n_seg = fatal(a) ? 0 : (int)a.counts[0];
  const int lane = threadIdx.x & 63;
  int32_t *wr = row[threadIdx.x >> 6];
  const int64_t n_ch = (n_out + kTgtChunk - 1) / kTgtChunk;
  const int64_t nw = (int64_t)gridDim.x * (kBlock / 64);
  // the next chunk's bitmask half and offset are loaded while this one's
  // targets are placed and stored
  int64_t ch = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  uint64_t word = 0;
  int32_t off = 0;
  if (ch < n_ch) {
    word = a.tbits[ch * (kTgtChunk / 64) + lane / 2];
    off = a.chunk_off[ch];
  }
  for (; ch < n_ch; ch += nw) {
    uint64_t next_word = 0;
    int32_t next_off = 0;
    if (ch + nw < n_ch) {
      next_word = a.tbits[(ch + nw) * (kTgtChunk / 64) + lane / 2];
      next_off = a.chunk_off[ch + nw];
    }
    uint32_t bits = (uint32_t)(word >> (32 * (lane & 1)));
    const int c = __popc(bits);
    int x = c;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    const int total = __shfl(x, 63, 64);
    const int32_t o0 = (int32_t)(ch * kTgtChunk + 32 * lane);
    int k = x - c;
    while (bits) {
      wr[k++] = o0 + __ffs(bits) - 1;
      bits &= bits - 1;
    }
    wave_lds_sync();
    for (int i = lane; i < total; i += 64) a.targets[off + i] = wr[i];
    wave_lds_sync();
    word = next_word;
    off = next_off;
  }
  const int n_mask = (int)a.counts[2];
  for (int s = blockIdx.x * kBlock + threadIdx.x; s <= n_seg; s += gridDim.x * kBlock) {
    const int64_t o = a.cu_seqlens[s];
    int v = n_mask;
    if (o < n_out) {
      const int64_t ch = o / kTgtChunk;
      v = a.chunk_off[ch];
      const uint64_t *w = a.tbits + ch * (kTgtChunk / 64);
      const int64_t full = (o - ch * kTgtChunk) / 64;
      for (int64_t k = 0; k < full; ++k) v += __popcll(w[k]);
      const int rem = (int)(o % 64);
      if (rem) v += __popcll(w[full] & ((1ull << rem) - 1));
    }
    a.cu_targets[s] = v;
  }
}

// ---------------------------------------------------------------- text-level Match
// Match compares each aligned block's text key.  Keys never change while
// Algorithm 1 runs (a transfer copies a block with the same text), so the
// closed form above holds with "T_j <= T_i" read as: T_i has at least as many
// blocks and the first |T_j| keys agree.  Transfers may change block lengths:
// a survivor block carries the tokens of one source block (its own, or the
// block of the largest absorbed timeline with an llm block there), and the
// output is laid out from the chosen blocks' lengths.
AJ_DEV bool llm_block(const MergeArgs &a, int b) {
  return (a.flags[a.blk_start[b]] & AJ_AUTHOR_MASK) == AJ_AUTHOR_LLM;
}

// Largest index b in [lo, hi] with off[b] <= v (off ascending, off[lo] <= v).
AJ_DEV int upper_index(const int32_t *off, int64_t v, int lo, int hi) {
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (off[mid] <= v) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Block starts per chunk of kChunk tokens.
__global__ __launch_bounds__(kBlock) void blk_count_kernel(MergeArgs a) {
  const int64_t u0 = (int64_t)blockIdx.x * kChunk + threadIdx.x * 4;
  int c = 0;
#pragma unroll
  for (int r = 0; r < 4; ++r)
    c += (u0 + r < a.n_tok) && (a.flags[u0 + r] & AJ_FLAG_BLOCK_START);
  int tot;
  block_scan_incl<kBlock>(c, &tot);
  if (threadIdx.x == 0) a.chunk_cnt[blockIdx.x] = tot;
}

// blk_start[b] = first token of block b (the scan checked there are n_blk).
__global__ __launch_bounds__(kBlock) void blk_write_kernel(MergeArgs a) {
  if (fatal(a)) return;
  const int64_t u0 = (int64_t)blockIdx.x * kChunk + threadIdx.x * 4;
  int f[4], c = 0;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    f[r] = (u0 + r < a.n_tok) && (a.flags[u0 + r] & AJ_FLAG_BLOCK_START);
    c += f[r];
  }
  int tot;
  int incl = block_scan_incl<kBlock>(c, &tot);
  int w = a.chunk_off[blockIdx.x] + incl - c;
#pragma unroll
  for (int r = 0; r < 4; ++r)
    if (f[r]) a.blk_start[w++] = (int32_t)(u0 + r);
  if (blockIdx.x == 0 && threadIdx.x == 0) a.blk_start[a.n_blk] = (int32_t)a.n_tok;
}

// tl_blk[i] = the block that starts at timeline i's first token.
__global__ void tl_blk_kernel(MergeArgs a) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i > a.n_tl || fatal(a)) return;
  if (i == a.n_tl) { a.tl_blk[i] = a.n_blk; return; }
  const int64_t u = a.tl_tok_off[i];
  int lo = 0, hi = a.n_blk;          // first block starting at or after u
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if (a.blk_start[mid] < u) lo = mid + 1; else hi = mid;
  }
  if (lo == a.n_blk || a.blk_start[lo] != u) raise(a, AJ_DEVERR_BLOCKS);
  a.tl_blk[i] = lo;
}

__global__ void blk_tl_kernel(MergeArgs a) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= a.n_blk || fatal(a)) return;
  a.blk_tl[b] = upper_index(a.tl_blk, b, 0, a.n_tl - 1);
  a.blk_claim[b] = -1;
  a.dst_off[b] = -1;
}

// One wavefront per timeline j: candidates from the episode's last timeline
// down, key comparison with early exit.
__global__ __launch_bounds__(64) void find_absorber_text_kernel(MergeArgs a) {
  const int j = blockIdx.x;
  if (fatal(a)) {
    if (threadIdx.x == 0) a.absorber[j] = -1;
    return;
  }
  int lo = 0, hi = a.n_traj - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (a.traj_tl_off[mid] <= j) lo = mid; else hi = mid - 1;
  }
  while (lo + 1 < a.n_traj && a.traj_tl_off[lo + 1] <= j) ++lo;
  const int last = a.traj_tl_off[lo + 1] - 1;
  const int bj = a.tl_blk[j], nj = a.tl_blk[j + 1] - bj;
  int result = -1;
  for (int i = last; i > j; --i) {
    const int bi = a.tl_blk[i];
    if (a.tl_blk[i + 1] - bi < nj) continue;
    bool equal = true;
    for (int k0 = 0; k0 < nj; k0 += 64) {
      const int k = k0 + (int)threadIdx.x;
      const bool bad = k < nj && a.blk_text[bj + k] != a.blk_text[bi + k];
      if (__ballot(bad)) { equal = false; break; }
    }
    if (equal) { result = i; break; }
  }
  if (threadIdx.x == 0) a.absorber[j] = result;
}

// llm blocks of absorbed timelines vote for the survivor block they align with.
__global__ void claim_text_kernel(MergeArgs a) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= a.n_blk || fatal(a)) return;
  const int t = a.blk_tl[b];
  const int s = a.absorber[t];
  if (s < 0 || !llm_block(a, b)) return;
  atomicMax(&a.blk_claim[a.tl_blk[s] + (b - a.tl_blk[t])], t);
}

// Source block and output length of every block (0 for absorbed timelines).
__global__ void select_text_kernel(MergeArgs a) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= a.n_blk || fatal(a)) return;
  const int t = a.blk_tl[b];
  int src = -1;
  if (a.absorber[t] < 0) {
    src = b;
    const int c = a.blk_claim[b];
    if (!llm_block(a, b) && c >= 0) src = a.tl_blk[c] + (b - a.tl_blk[t]);
  }
  a.src_blk[b] = src;
  a.blk_off[b] = src >= 0 ? a.blk_start[src + 1] - a.blk_start[src] : 0;
}

// Single workgroup of 1024 threads: output offsets of the blocks (exclusive
// scan of their lengths, in place), then the survivor scan as in resolve.
__global__ __launch_bounds__(1024) void resolve_text_kernel(MergeArgs a) {
  __shared__ int carry_seg, carry_tok, carry_max;
  if (threadIdx.x == 0) { carry_seg = 0; carry_tok = 0; carry_max = 0; }
  __syncthreads();
  const bool bad = fatal(a);
  if (!bad) {
    for (int base = 0; base < a.n_blk; base += 1024) {
      const int b = base + threadIdx.x;
      const int len = b < a.n_blk ? a.blk_off[b] : 0;
      int tot;
      const int incl = block_scan_incl<1024>(len, &tot);
      if (b < a.n_blk) a.blk_off[b] = carry_tok + incl - len;
      __syncthreads();
      if (threadIdx.x == 0) carry_tok += tot;
      __syncthreads();
    }
    if (threadIdx.x == 0) a.blk_off[a.n_blk] = carry_tok;
  }
  // the block offsets written above are read back by other threads
  __syncthreads();
  for (int base = 0; base < a.n_tl; base += 1024) {
    const int i = base + threadIdx.x;
    const int surv = !bad && i < a.n_tl && a.absorber[i] < 0;
    int tot_s;
    const int is = block_scan_incl<1024>(surv, &tot_s);
    if (i < a.n_tl) {
      if (surv) {
        const int seg = carry_seg + is - 1;
        const int o0 = a.blk_off[a.tl_blk[i]];
        a.tl_seg[i] = seg;
        a.seg_src[seg] = i;
        a.cu_seqlens[seg] = o0;
        atomicMax(&carry_max, a.blk_off[a.tl_blk[i + 1]] - o0);
      } else {
        a.tl_seg[i] = -1;
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) carry_seg += tot_s;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const int n_out = bad ? 0 : carry_tok;
    a.cu_seqlens[carry_seg] = n_out;
    a.counts[0] = carry_seg;
    a.counts[1] = n_out;
    a.counts[2] = 0;
    a.counts[3] = carry_max;
  }
}

// Where each chosen source block lands.
__global__ void place_text_kernel(MergeArgs a) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= a.n_blk || fatal(a)) return;
  const int src = a.src_blk[b];
  if (src < 0) return;
  const int o = a.blk_off[b];
  a.dst_off[src] = o;
  a.dst_pos[src] = o - a.blk_off[a.tl_blk[a.blk_tl[b]]];
}

// One thread per input token: copy it to where its block lands, if anywhere.
__global__ __launch_bounds__(kBlock) void emit_text_kernel(MergeArgs a) {
  if (fatal(a)) return;
  const int64_t u0 = (int64_t)blockIdx.x * blockDim.x;
  __shared__ int r[2];
  if (threadIdx.x == 0) {
    int64_t u1 = u0 + blockDim.x - 1;
    if (u1 >= a.n_tok) u1 = a.n_tok - 1;
    r[0] = upper_index(a.blk_start, u0, 0, a.n_blk - 1);
    r[1] = upper_index(a.blk_start, u1, r[0], a.n_blk - 1);
  }
  __syncthreads();
  const int64_t u = u0 + threadIdx.x;
  if (u >= a.n_tok) return;
  if ((a.flags[u] & AJ_AUTHOR_MASK) == AJ_AUTHOR_MASK) raise(a, AJ_DEVERR_BAD_FLAGS);
  const int b = upper_index(a.blk_start, u, r[0], r[1]);
  const int o0 = a.dst_off[b];
  if (o0 < 0) return;
  const int p = (int)(u - a.blk_start[b]);
  const bool llm = llm_block(a, b);
  a.otok[o0 + p] = a.tok[u];
  a.opos[o0 + p] = a.dst_pos[b] + p;
  a.omask[o0 + p] = llm;
  a.olp[o0 + p] = llm ? a.old_logprob[u] : 0.f;
  a.oadv[o0 + p] = llm ? a.adv[u] : 0.f;
}

// One wavefront per block: an llm block of the output whose tokens before it
// in its segment differ from those before it in its own timeline.
__global__ __launch_bounds__(64) void ti_kernel(MergeArgs a) {
  const int b = blockIdx.x;
  if (fatal(a)) return;
  const int src = a.src_blk[b];
  if (src < 0 || !llm_block(a, src)) return;
  const int o1 = a.blk_off[b];
  const int o0 = a.blk_off[a.tl_blk[a.blk_tl[b]]];
  const int64_t u1 = a.blk_start[src];
  const int64_t u0 = a.tl_tok_off[a.blk_tl[src]];
  bool drift = (int64_t)(o1 - o0) != u1 - u0;
  for (int64_t q0 = 0; !drift && q0 < o1 - o0; q0 += 64 * 4) {
    bool bad = false;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t q = q0 + r * 64 + threadIdx.x;
      if (q < o1 - o0) bad |= a.otok[o0 + q] != a.tok[u0 + q];
    }
    drift = __ballot(bad) != 0;
  }
  if (drift && threadIdx.x == 0) {
    atomicAdd((unsigned long long *)&a.ti[0], 1ull);
    atomicAdd((unsigned long long *)&a.ti[1],
              (unsigned long long)(a.blk_start[src + 1] - a.blk_start[src]));
  }
}

struct MergeWs {
  int32_t *status, *tl_seg, *chunk_cnt, *chunk_off, *rblk, *tblk;
  int32_t n_rblk, n_tblk;
  uint64_t *tbits;
  int32_t n_slots;
  int32_t *ep_first, *ep_last, *cand, *miss, *rcnt, *runs;
  int4 *slot_rec;
  int32_t *seg_base, *range_rec;
  int32_t *blk_start, *tl_blk, *blk_tl, *blk_claim, *src_blk, *blk_off, *dst_off, *dst_pos;
  size_t bytes;
};

// n_blk < 0: token-level Match or no merge (no per-block arrays).
MergeWs carve(void *ws, int32_t n_tl, int64_t n_tok, int32_t n_blk = -1) {
  aj::Carver c(ws);
  MergeWs w{};
  int64_t n_chunks = (n_tok + kChunk - 1) / kChunk;
  auto at_least1 = [](int64_t n) { return n > 0 ? n : 1; };
  w.status = c.take<int32_t>(4);
  w.n_rblk = (int32_t)((n_tl + kResSpan - 1) / kResSpan);
  w.rblk = c.take<int32_t>(4 * at_least1(w.n_rblk));
  w.n_tblk = (int32_t)(((n_tok + kTgtChunk - 1) / kTgtChunk + kTgtScanSpan - 1) / kTgtScanSpan);
  w.tblk = c.take<int32_t>(at_least1(w.n_tblk));
  w.tl_seg = c.take<int32_t>(at_least1(n_tl));
  w.chunk_cnt = c.take<int32_t>(at_least1(n_chunks));
  w.chunk_off = c.take<int32_t>(at_least1(n_chunks));
  // one target bit per output; emit writes whole 2048-output spans
  w.tbits = c.take<uint64_t>((n_tok + kTgtChunk - 1) / kTgtChunk * (kTgtChunk / 64) + 1);
  w.seg_base = c.take<int32_t>(at_least1(n_tl));
  w.range_rec = c.take<int32_t>(at_least1((n_tok + kEmitSpan - 1) / kEmitSpan) * kRecInts);
  if (n_blk < 0) {
    // compare items: n_tok / kCmpChunk + n_tl slots (n_tok < 2^31)
    w.n_slots = (int32_t)(n_tok / kCmpChunk + n_tl);
    w.ep_first = c.take<int32_t>(at_least1(n_tl));
    w.ep_last = c.take<int32_t>(at_least1(n_tl));
    w.cand = c.take<int32_t>(at_least1(n_tl));
    w.miss = c.take<int32_t>(at_least1(n_tl));
    w.slot_rec = c.take<int4>(at_least1(w.n_slots));
    w.rcnt = c.take<int32_t>(at_least1(w.n_slots));
    w.runs = c.take<int32_t>(at_least1((int64_t)w.n_slots * 2 * kRuns));
  } else {
    w.blk_start = c.take<int32_t>(n_blk + 1);
    w.tl_blk = c.take<int32_t>((int64_t)n_tl + 1);
    w.blk_tl = c.take<int32_t>(at_least1(n_blk));
    w.blk_claim = c.take<int32_t>(at_least1(n_blk));
    w.src_blk = c.take<int32_t>(at_least1(n_blk));
    w.blk_off = c.take<int32_t>(n_blk + 1);
    w.dst_off = c.take<int32_t>(at_least1(n_blk));
    w.dst_pos = c.take<int32_t>(at_least1(n_blk));
  }
  w.bytes = c.bytes();
  return w;
}

int check_io(const aj_timelines *in, aj_packed *out, const char *name) {
  AJ_REQUIRE(in && out, AJ_ERR_NULL, "%s: null argument struct", name);
  AJ_REQUIRE(in->n_traj >= 0 && in->n_tl >= 0 && in->n_tok >= 0 && in->n_tok < (int64_t)1 << 31,
             AJ_ERR_SHAPE, "%s: n_traj=%d n_tl=%d n_tok=%lld out of range", name, in->n_traj,
             in->n_tl, (long long)in->n_tok);
  AJ_REQUIRE(in->n_tl == 0 || in->n_traj > 0, AJ_ERR_SHAPE, "%s: timelines without episodes", name);
  AJ_REQUIRE(in->traj_tl_off && in->tl_tok_off, AJ_ERR_NULL, "%s: null offsets", name);
  AJ_REQUIRE(in->n_tok == 0 || (in->tok && in->flags && in->old_logprob && in->adv), AJ_ERR_NULL,
             "%s: null token arrays", name);
  AJ_REQUIRE(out->absorber || in->n_tl == 0, AJ_ERR_NULL, "%s: null absorber", name);
  AJ_REQUIRE(out->cu_seqlens && out->seg_src && out->cu_targets && out->counts, AJ_ERR_NULL,
             "%s: null segment outputs", name);
  AJ_REQUIRE(in->n_tok == 0 || (out->tok && out->pos && out->mask && out->old_logprob &&
                                out->adv && out->targets),
             AJ_ERR_NULL, "%s: null token outputs", name);
  return AJ_OK;
}

MergeArgs make_args(const aj_timelines *in, aj_packed *out, int32_t *err, const MergeWs &w) {
  MergeArgs a{};
  a.n_traj = in->n_traj; a.n_tl = in->n_tl; a.n_tok = in->n_tok;
  a.traj_tl_off = in->traj_tl_off; a.tl_tok_off = in->tl_tok_off;
  a.tok = in->tok; a.flags = in->flags; a.old_logprob = in->old_logprob; a.adv = in->adv;
  a.absorber = out->absorber; a.cu_seqlens = out->cu_seqlens; a.seg_src = out->seg_src;
  a.cu_targets = out->cu_targets; a.counts = out->counts;
  a.otok = out->tok; a.opos = out->pos; a.omask = out->mask; a.olp = out->old_logprob;
  a.oadv = out->adv; a.targets = out->targets;
  a.status = w.status; a.tl_seg = w.tl_seg; a.tbits = w.tbits;
  a.n_slots = w.n_slots; a.ep_first = w.ep_first; a.ep_last = w.ep_last; a.cand = w.cand;
  a.miss = w.miss; a.slot_rec = w.slot_rec; a.rcnt = w.rcnt; a.runs = w.runs;
  a.seg_base = w.seg_base; a.range_rec = w.range_rec;
  a.chunk_cnt = w.chunk_cnt; a.chunk_off = w.chunk_off; a.user_err = err;
  a.rblk = w.rblk; a.n_rblk = w.n_rblk; a.tblk = w.tblk; a.n_tblk = w.n_tblk;
  a.blk_start = w.blk_start; a.tl_blk = w.tl_blk; a.blk_tl = w.blk_tl; a.blk_claim = w.blk_claim;
  a.src_blk = w.src_blk; a.blk_off = w.blk_off; a.dst_off = w.dst_off; a.dst_pos = w.dst_pos;
  return a;
}

// The call's status word, cleared, then the input checks on a grid.
void launch_validate(const MergeArgs &a, hipStream_t s) {
  const int n_val = (a.n_tl > a.n_traj ? a.n_tl : a.n_traj) + 1;
  init_status_kernel<<<1, 64, 0, s>>>(a);
  validate_kernel<<<(n_val + kBlock - 1) / kBlock, kBlock, 0, s>>>(a);
}

// Workgroups of kBlock threads of a grid-stride kernel that are resident on
// the current device at once (its occupancy times the CU count), so the
// stride loop runs in one round; looked up once per device and kernel.
constexpr int kMaxDev = 64;
int resident_wgs(const void *kernel, int slot) {
  static std::mutex mu;
  static int cache[kMaxDev][2];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev) return kEmitWgs;
  std::lock_guard<std::mutex> lk(mu);
  if (!cache[dev][slot]) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kBlock, 0) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        per_cu <= 0 || cus <= 0)
      return kEmitWgs;
    cache[dev][slot] = per_cu * cus;
  }
  return cache[dev][slot];
}

// The target list and per-segment target offsets, once tok/pos/mask are out.
// counted: emit already wrote the per-chunk target counts and the bitmask.
void launch_targets(const MergeArgs &a, hipStream_t s, bool counted) {
  const int64_t n_chunks = (a.n_tok + kTgtChunk - 1) / kTgtChunk;
  if (a.n_tok > 0 && !counted) tgt_count_kernel<<<n_chunks, kBlock, 0, s>>>(a);
  tgt_offsets_kernel<<<a.n_tblk > 0 ? a.n_tblk : 1, kBlock, 0, s>>>(a);
  const int64_t segs = ((int64_t)a.n_tl + 1 + kBlock - 1) / kBlock;
  const int64_t g = n_chunks > segs ? n_chunks : segs;
  const int64_t gw = resident_wgs(reinterpret_cast<const void *>(tgt_write_kernel), 1);
  tgt_write_kernel<<<(int)(g < gw ? g : gw), kBlock, 0, s>>>(a);
}

int run(const aj_timelines *in, aj_packed *out, int32_t *err, void *ws, size_t ws_bytes,
        void *stream, bool merge) {
  const char *name = merge ? "aj_merge_timelines" : "aj_flatten_timelines";
  if (int rc = check_io(in, out, name)) return rc;
  MergeWs w = carve(ws, in->n_tl, in->n_tok);
  AJ_REQUIRE(ws, AJ_ERR_NULL, "%s: null workspace", name);
  AJ_REQUIRE(ws_bytes >= w.bytes, AJ_ERR_WORKSPACE, "%s: workspace %zu < %zu bytes", name,
             ws_bytes, w.bytes);
  MergeArgs a = make_args(in, out, err, w);

  hipStream_t s = (hipStream_t)stream;
  const int tk = aj::timing_begin(s, AJ_KC_MERGE, 0.0);
  if (merge) {
    // the checks and the per-timeline tables, then Algorithm 1 in closed form
    const int n_set = (in->n_tl > in->n_traj ? in->n_tl : in->n_traj) + 1;
    init_status_kernel<<<1, 64, 0, s>>>(a);
    setup_kernel<<<(n_set + kBlock - 1) / kBlock, kBlock, 0, s>>>(a);
    if (in->n_tl > 0) {
      filter_kernel<<<(in->n_tl + kBlock / 64 - 1) / (kBlock / 64), kBlock, 0, s>>>(a);
      if (a.n_slots > 0) compare_kernel<<<a.n_slots, kBlock, 0, s>>>(a);
      finalize_kernel<<<(in->n_tl + kFinPer - 1) / kFinPer, kBlock, 0, s>>>(a);
    }
  } else {
    launch_validate(a, s);
    if (in->n_tl > 0) fill_absorber_kernel<<<(in->n_tl + kBlock - 1) / kBlock, kBlock, 0, s>>>(a);
  }
  resolve_kernel<<<a.n_rblk > 0 ? a.n_rblk : 1, kBlock, 0, s>>>(a);
  if (in->n_tok > 0) {
    const int64_t spans = (in->n_tok + kEmitSpan - 1) / kEmitSpan;
    range_kernel<<<(int)((spans + kBlock / 64 - 1) / (kBlock / 64)), kBlock, 0, s>>>(a, merge ? 1 : 0);
    const int64_t gw = resident_wgs(reinterpret_cast<const void *>(emit_kernel), 0);
    emit_kernel<<<(int)(spans < gw ? spans : gw), kBlock, 0, s>>>(a, merge ? 1 : 0);
  }
  launch_targets(a, s, true);
  aj::timing_end(s, tk);
  return aj::check_launch(name);
}

int run_text(const aj_timelines *in, const aj_block_texts *text, aj_packed *out, int64_t *ti,
             int32_t *err, void *ws, size_t ws_bytes, void *stream) {
  const char *name = "aj_merge_timelines_text";
  if (int rc = check_io(in, out, name)) return rc;
  AJ_REQUIRE(text, AJ_ERR_NULL, "%s: null text keys", name);
  AJ_REQUIRE(text->n_blk >= 0 && text->n_blk <= in->n_tok, AJ_ERR_SHAPE,
             "%s: n_blk=%d outside [0, n_tok=%lld] (blocks are never empty)", name, text->n_blk,
             (long long)in->n_tok);
  AJ_REQUIRE(text->n_blk == 0 || text->key, AJ_ERR_NULL, "%s: null key array", name);
  MergeWs w = carve(ws, in->n_tl, in->n_tok, text->n_blk);
  AJ_REQUIRE(ws, AJ_ERR_NULL, "%s: null workspace", name);
  AJ_REQUIRE(ws_bytes >= w.bytes, AJ_ERR_WORKSPACE, "%s: workspace %zu < %zu bytes", name,
             ws_bytes, w.bytes);
  MergeArgs a = make_args(in, out, err, w);
  a.n_blk = text->n_blk;
  a.blk_text = text->key;
  a.ti = ti;

  const int n_blk = text->n_blk;
  const int64_t n_chunks = (in->n_tok + kChunk - 1) / kChunk;
  const int gblk = (n_blk + kBlock - 1) / kBlock;
  hipStream_t s = (hipStream_t)stream;
  const int tk = aj::timing_begin(s, AJ_KC_MERGE, 0.0);
  launch_validate(a, s);
  // blocks: first tokens, first block per timeline, timeline per block
  if (in->n_tok > 0) blk_count_kernel<<<n_chunks, kBlock, 0, s>>>(a);
  blk_scan_kernel<<<1, 1024, 0, s>>>(a, (int)n_chunks);
  if (in->n_tok > 0) blk_write_kernel<<<n_chunks, kBlock, 0, s>>>(a);
  tl_blk_kernel<<<(in->n_tl + 1 + kBlock - 1) / kBlock, kBlock, 0, s>>>(a);
  if (n_blk > 0) blk_tl_kernel<<<gblk, kBlock, 0, s>>>(a);
  // Algorithm 1 in closed form on the keys, then the chosen blocks
  if (in->n_tl > 0) find_absorber_text_kernel<<<in->n_tl, 64, 0, s>>>(a);
  if (n_blk > 0) {
    claim_text_kernel<<<gblk, kBlock, 0, s>>>(a);
    select_text_kernel<<<gblk, kBlock, 0, s>>>(a);
  }
  resolve_text_kernel<<<1, 1024, 0, s>>>(a);
  if (n_blk > 0) place_text_kernel<<<gblk, kBlock, 0, s>>>(a);
  if (in->n_tok > 0)
    emit_text_kernel<<<(in->n_tok + kBlock - 1) / kBlock, kBlock, 0, s>>>(a);
  launch_targets(a, s, false);
  if (ti && n_blk > 0) ti_kernel<<<n_blk, 64, 0, s>>>(a);
  aj::timing_end(s, tk);
  return aj::check_launch(name);
}

}  // namespace

extern "C" size_t aj_merge_workspace_bytes(int32_t n_traj, int32_t n_tl, int64_t n_tok) {
  (void)n_traj;
  return carve(nullptr, n_tl, n_tok).bytes;
}

extern "C" size_t aj_merge_text_workspace_bytes(int32_t n_traj, int32_t n_tl, int64_t n_tok,
                                                int32_t n_blk) {
  (void)n_traj;
  return carve(nullptr, n_tl, n_tok, n_blk < 0 ? 0 : n_blk).bytes;
}

extern "C" int aj_merge_timelines_text(const aj_timelines *in, const aj_block_texts *text,
                                       aj_packed *out, int64_t *ti, int32_t *err, void *ws,
                                       size_t ws_bytes, void *stream) {
  return run_text(in, text, out, ti, err, ws, ws_bytes, stream);
}

extern "C" int aj_merge_timelines(const aj_timelines *in, aj_packed *out, int32_t *err, void *ws,
                                  size_t ws_bytes, void *stream) {
  return run(in, out, err, ws, ws_bytes, stream, true);
}

extern "C" int aj_flatten_timelines(const aj_timelines *in, aj_packed *out, int32_t *err,
                                    void *ws, size_t ws_bytes, void *stream) {
  return run(in, out, err, ws, ws_bytes, stream, false);
}

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

// Device address of `scratch` on the current device, looked up once per device.
int scratch_ptr(void **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return aj::fail(AJ_ERR_HIP, "aj_merge_timelines_noalloc: no current device (%d)", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return aj::fail(AJ_ERR_HIP, "aj_merge_timelines_noalloc: hipGetSymbolAddress: %s",
                      hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return AJ_OK;
}
}  // namespace

extern "C" size_t aj_merge_noalloc_max_workspace_bytes(void) { return kScratchBytes; }

extern "C" int aj_merge_timelines_noalloc(const aj_timelines *in, aj_packed *out, int32_t *err,
                                          void *stream) {
  AJ_REQUIRE(in, AJ_ERR_NULL, "aj_merge_timelines_noalloc: null input");
  const size_t need = carve(nullptr, in->n_tl, in->n_tok).bytes;
  AJ_REQUIRE(need <= kScratchBytes, AJ_ERR_WORKSPACE,
             "aj_merge_timelines_noalloc: %d timelines of %lld tokens need %zu bytes of "
             "workspace, more than the built-in %zu",
             in->n_tl, (long long)in->n_tok, need, kScratchBytes);
  void *ws = nullptr;
  if (int rc = scratch_ptr(&ws)) return rc;
  return run(in, out, err, ws, kScratchBytes, stream, true);
}

extern "C" int aj_plan_packs(const int32_t *cu_seqlens, int32_t n_seg, int32_t max_tokens,
                             int32_t *pack_seg_off, int32_t *n_packs) {
  AJ_REQUIRE(cu_seqlens && pack_seg_off && n_packs, AJ_ERR_NULL, "aj_plan_packs: null pointer");
  AJ_REQUIRE(n_seg >= 0 && max_tokens > 0, AJ_ERR_SHAPE, "aj_plan_packs: n_seg=%d max_tokens=%d",
             n_seg, max_tokens);
  for (int s = 0; s < n_seg; ++s)
    AJ_REQUIRE(cu_seqlens[s] <= cu_seqlens[s + 1], AJ_ERR_SHAPE,
               "aj_plan_packs: cu_seqlens not monotone at %d", s);
  int np = 0;
  int s = 0;
  while (s < n_seg) {
    pack_seg_off[np++] = s;
    const int32_t start = cu_seqlens[s];
    int e = s + 1;
    while (e < n_seg && cu_seqlens[e + 1] - start <= max_tokens) ++e;
    s = e;
  }
  pack_seg_off[np] = n_seg;
  *n_packs = np;
  return AJ_OK;
}
