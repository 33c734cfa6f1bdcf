// Global top-W beam selection (Sec. 2.1) on gfx950.
//
// Every live beam p of a request is expanded over the V codebook entries; the
// candidate (p, v) has score  beam[p] + logp[p][v]  (one fp32 rounding; logp
// alone when no beam scores are given) and flat index p * V + v.  The W best
// candidates are kept, best first.  The order is total: higher score first,
// equal scores by lower flat index, -0.0 below +0.0, every NaN below every
// number.  It is realised on an unsigned 32-bit key that is monotone in the
// score (sign-magnitude flip; all NaNs map to 0), then on the flat index.
//
// The work is HBM-bound (N = W_prev * V fp32 scores per request, read once),
// so it is organised as filters with provable bounds rather than a global
// sort.  Large calls whose workgroups all fit the device at once take the
// one-pass path (each chunk held in registers from its single read while a
// bound forms across workgroups, then a placing launch; described at its
// kernels below); other large calls the two-pass path (wave maxima, then one
// filter pass, then the one-pass path's placing launch, or ranking
// workgroups per request beyond 512 chunks); smaller ones a reduction tree.  A 512-thread workgroup holds 16384 candidates (32 per lane):
//   * stage kernel: keeps a superset of its candidates' top min(W, n) and
//     writes it, in index order, to an output slot of `cap` (key, index)
//     pairs plus a count.  A 2048-bin histogram of the maxima of groups of
//     4 consecutive slots of a lane gives a key that at least need of the
//     candidates reach; everything below it is dropped, so no member of the
//     top need is lost and about need survive.  When the survivors do not
//     fit the slot, the exact cut is taken instead (radix select over the
//     workgroup).
//   * final kernel: one workgroup per request filters the last <= 16384
//     candidates the same way, sorts the survivors (a stable LSD radix sort
//     on the score key; they arrive in index order, so ties stay in index
//     order) and writes the first W.
// The stage input of stage s >= 1 is the slot array of stage s - 1; a
// workgroup reads 16384 / cap consecutive slots.  Slots hold increasing index
// ranges, so position order inside a workgroup is index order, which is what
// the tie rule needs.
#include <algorithm>
#include <mutex>

#include "internal.h"

// Device scratch of the allocation-free entry point (onela_select_beams_noalloc):
// the workspace of a selection call, held by every GPU the library runs on
// until the process ends.  Host code never uses this name as an address (in
// host code it is a host-side stand-in): the device address comes from
// hipGetSymbolAddress, once per device, in select_scratch below.
static __device__ __align__(256) unsigned char scratch[onela::kSelectScratchBytes];

namespace onela {
namespace {

constexpr int kThreads = kSelectThreads;
constexpr int kWaves = kThreads / 64;
constexpr int kNI = kSelectChunk / kThreads;  // candidates per lane
constexpr int kSortCap = 4096;                // survivors the final kernel sorts
constexpr int kMaxSlotsPerGroup = 256;
constexpr int kRankCap = 4096;                // survivors the rank kernel orders
constexpr int kRankPer = kThreads / 16;       // survivors ranked per workgroup (16 lanes each)
constexpr int kRankBlocks = kRankCap / kRankPer;
constexpr int kOnePassRankMax = 1024;         // widest result of the one-pass path
constexpr int kOnePassFinalParts = 64;       // workgroups per request placing survivors (at most)
constexpr int kOnePassSegPer = 8;             // wave summaries per thread of the bound:
                                              // chunks <= kOnePassSegPer * kThreads / 8
static_assert(kNI == 32, "validity masks are 32-bit");

struct SelectParams {
  const float* logp;        // [R][N] log-probabilities, N = W_prev * V
  const float* beam;        // [R][W_prev] beam scores, or null
  const uint2* cand_in;     // [R][nslots_in][cap] (key, flat index); null: read logp
  const unsigned* cnt_in;   // [R][nslots_in] counts (two-pass: (count, largest key) pairs)
  uint2* cand_out;          // [R][nwg][cap]        (stage kernel)
  unsigned* cnt_out;        // [R][nwg] counts (two-pass: (count, largest key) pairs)
  int* parents;             // [R][W]               (final kernel)
  int* tokens;
  float* scores;
  unsigned N, V, W_prev, W;
  unsigned cap, lcap;       // slot capacity (a power of two) and its log2
  unsigned group;           // input slots per workgroup (16384 / cap)
  unsigned nslots_in;       // input slots per request (slot input)
  unsigned* segmax;         // [R][nseg] largest key of each wave's candidates (two-pass)
  unsigned nseg;
  unsigned nwg;             // workgroups per request
  double inv_v;             // 1 / V
  // one-pass path
  struct OnePassCtl* ctl;   // call counter and per-request bound words
  uint4* ex;                // [R][nseg] per wave: (M, m, kM, check), see the one-pass path
  unsigned long long wait_ticks;  // how long a workgroup waits for the bound (wall clock)
  unsigned fparts;          // workgroups per request of the final kernel
  // two-pass path with a bound word per request (see select_summary_kernel)
  unsigned long long* tp_bound;  // [R] (c* + 1) << 32 | B, or null: the filter forms the bound
};

// Cross-workgroup state of the one-pass path, at the start of the workspace
// (zero-filled before the first call).  The bound words are zero when a call
// starts, and the call's final kernel zeroes its requests' words again; the
// epoch counts the calls (see the summaries' tags).
struct OnePassCtl {
  unsigned epoch;     // this call's tag is epoch + 1
  unsigned pad_[3];
  unsigned long long bound[kSelectOnePassMaxRequests];  // (1 << 32) | bound, once known
  // two-pass summary pass: workgroups of each request that have published
  // their summaries (zero between calls: the last one returns it to zero)
  unsigned arrive[kSelectOnePassMaxRequests];
};
static_assert(sizeof(OnePassCtl) <= kSelectCtlBytes, "control block fits its region");

struct alignas(16) SelShared {
  unsigned hist[2048];  // exact cut: one 2048-bin histogram; bound: 8 x 256 bins
  unsigned tab[kNI * kWaves + 4];
  unsigned red[2][kWaves];
  unsigned scnt[kMaxSlotsPerGroup];
  unsigned digit, need, cnt;
};

// ---- wave-level helpers (DPP) ----------------------------------------------

template <int CTRL, int ROWS = 0xF>
__device__ inline unsigned dppu(unsigned x) {
  return unsigned(__builtin_amdgcn_update_dpp(0, int(x), CTRL, ROWS, 0xF, false));
}

__device__ inline unsigned lane_id() { return threadIdx.x & 63; }

__device__ inline unsigned mbcnt(unsigned long long m) {
  return __builtin_amdgcn_mbcnt_hi(unsigned(m >> 32), __builtin_amdgcn_mbcnt_lo(unsigned(m), 0u));
}

// Inclusive prefix sum over the 64 lanes.
__device__ inline unsigned wave_scan(unsigned x) {
  x += dppu<0x111>(x);       // row_shr:1
  x += dppu<0x112>(x);       // row_shr:2
  x += dppu<0x114>(x);       // row_shr:4
  x += dppu<0x118>(x);       // row_shr:8
  x += dppu<0x142, 0xA>(x);  // row_bcast:15 into rows 1, 3
  x += dppu<0x143, 0xC>(x);  // row_bcast:31 into rows 2, 3
  return x;
}

// (sum, min, max) over the 64 lanes, wave-uniform.
struct Red3 {
  unsigned sum, lo, hi;
};
__device__ inline Red3 wave_reduce(unsigned s, unsigned lo, unsigned hi) {
#define ONELA_RED_STEP(C)            \
  {                                  \
    s += dppu<C>(s);                 \
    lo = min(lo, dppu<C>(lo));       \
    hi = max(hi, dppu<C>(hi));       \
  }
  ONELA_RED_STEP(0xB1)   // quad_perm [1,0,3,2]
  ONELA_RED_STEP(0x4E)   // quad_perm [2,3,0,1]
  ONELA_RED_STEP(0x141)  // row_half_mirror
  ONELA_RED_STEP(0x140)  // row_mirror
#undef ONELA_RED_STEP
  Red3 r{0u, ~0u, 0u};
#pragma unroll
  for (int row = 0; row < 4; ++row) {
    r.sum += unsigned(__builtin_amdgcn_readlane(int(s), 16 * row));
    r.lo = min(r.lo, unsigned(__builtin_amdgcn_readlane(int(lo), 16 * row)));
    r.hi = max(r.hi, unsigned(__builtin_amdgcn_readlane(int(hi), 16 * row)));
  }
  return r;
}

// Bitwise OR over the 64 lanes, wave-uniform.
__device__ inline unsigned wave_or(unsigned x) {
  x |= dppu<0xB1>(x);   // quad_perm [1,0,3,2]
  x |= dppu<0x4E>(x);   // quad_perm [2,3,0,1]
  x |= dppu<0x141>(x);  // row_half_mirror
  x |= dppu<0x140>(x);  // row_mirror
  return unsigned(__builtin_amdgcn_readlane(int(x), 0)) |
         unsigned(__builtin_amdgcn_readlane(int(x), 16)) |
         unsigned(__builtin_amdgcn_readlane(int(x), 32)) |
         unsigned(__builtin_amdgcn_readlane(int(x), 48));
}

// (sum, min, max) over the workgroup.
__device__ inline Red3 block_reduce(SelShared& sh, unsigned s, unsigned lo, unsigned hi) {
  const Red3 w = wave_reduce(s, lo, hi);
  const unsigned wv = threadIdx.x >> 6;
  if (lane_id() == 0) {
    sh.tab[wv] = w.sum;
    sh.red[0][wv] = w.lo;
    sh.red[1][wv] = w.hi;
  }
  __syncthreads();
  Red3 r{0u, ~0u, 0u};
#pragma unroll
  for (int i = 0; i < kWaves; ++i) {
    r.sum += sh.tab[i];
    r.lo = min(r.lo, sh.red[0][i]);
    r.hi = max(r.hi, sh.red[1][i]);
  }
  __syncthreads();
  return r;
}

// x >> s for 0 <= s <= 32 (a shift by 32 gives 0).
__device__ inline unsigned shr(unsigned x, int s) {
  return unsigned(static_cast<unsigned long long>(x) >> s);
}

// Buffer resource of `bytes` bytes at `base` (a workgroup-uniform base; byte
// offsets stay below 2^31).  An access at or beyond `bytes` touches no
// memory (a load returns zeros), which lets a variable number of loads issue
// without a branch: a load under a branch is waited for where the branch
// joins, which serialises loads that should be in flight together.
__device__ inline __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, int bytes = 0x7fffffff) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0), bytes,
                                           0x00020000);
}

// ---- keys ------------------------------------------------------------------

// Monotone key of an fp32 score: larger score -> larger key, -0 < +0, every
// NaN -> 0 (below -inf, whose key is 0x007fffff).
__device__ inline unsigned order_key(float x) {
  const unsigned u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Row (beam) of a flat index: the fp64 quotient is within 1/V of the true
// one, so one correction step makes it exact.
__device__ inline unsigned row_of(unsigned idx, unsigned V, double inv_v) {
  unsigned p = unsigned(double(idx) * inv_v);
  if ((p + 1) * V <= idx) ++p;
  else if (p * V > idx) --p;
  return p;
}

// ---- index-ordered compaction ----------------------------------------------

// Ranks of the flagged elements (bit i of f: slot i) in position order, slot i
// of a lane sitting at position i * kThreads + threadIdx.x.  plan() takes the
// ballots and scans the 256 (slot, wave) counts; apply() calls fn(i, rank).
// The caller puts a barrier between apply() and the next use of sh.tab.
struct Ordered {
  unsigned pre[kNI / 4];  // wave-local ranks, 8 bits each
  unsigned total;
};

__device__ inline Ordered ordered_plan(unsigned f, SelShared& sh) {
  Ordered o;
  const unsigned lane = lane_id(), w = threadIdx.x >> 6;
  // slots flagged anywhere in the wave (a filter pass flags few): the others
  // skip their ballot
  const unsigned any = wave_or(f);
#pragma unroll
  for (int i = 0; i < kNI; ++i) {
    unsigned m = 0u, c = 0u;
    if ((any >> i) & 1u) {
      const unsigned long long b = __ballot((f >> i) & 1u);
      m = mbcnt(b);
      c = unsigned(__popcll(b));
    }
    o.pre[i / 4] = (i % 4 == 0) ? m : (o.pre[i / 4] | (m << (8 * (i % 4))));
    if (lane == 0) sh.tab[i * kWaves + w] = c;
  }
  __syncthreads();
  if (w == 0) {
    const uint4 v = reinterpret_cast<const uint4*>(sh.tab)[lane];
    const unsigned s = v.x + v.y + v.z + v.w;
    const unsigned inc = wave_scan(s);
    const unsigned ex = inc - s;
    reinterpret_cast<uint4*>(sh.tab)[lane] =
        make_uint4(ex, ex + v.x, ex + v.x + v.y, ex + v.x + v.y + v.z);
    if (lane == 63) sh.tab[kNI * kWaves] = inc;
  }
  __syncthreads();
  o.total = sh.tab[kNI * kWaves];
  return o;
}

template <typename F>
__device__ inline void ordered_apply(unsigned f, const Ordered& o, SelShared& sh, F&& fn) {
  const unsigned w = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < kNI; ++i)
    if ((f >> i) & 1u) fn(i, sh.tab[i * kWaves + w] + ((o.pre[i / 4] >> (8 * (i % 4))) & 0xffu));
}

// Ordered compaction for a filter that keeps few elements: only the slots
// that some lane of the wave flags are visited (wave-uniform loops over the
// set bits of the wave's OR).  sh.tab must be zero on entry (the counts of
// the slots no wave visits).  Returns the flagged count; apply_sparse() calls
// fn(i, rank) as ordered_apply() does.
__device__ inline unsigned ordered_plan_sparse(unsigned f, SelShared& sh) {
  const unsigned lane = lane_id(), w = threadIdx.x >> 6;
  for (unsigned any = wave_or(f); any != 0u; any &= any - 1u) {
    const int i = __builtin_ctz(any);
    const unsigned long long b = __ballot((f >> i) & 1u);
    if (lane == 0) sh.tab[i * kWaves + w] = unsigned(__popcll(b));
  }
  __syncthreads();
  if (w == 0) {
    const uint4 v = reinterpret_cast<const uint4*>(sh.tab)[lane];
    const unsigned s = v.x + v.y + v.z + v.w;
    const unsigned inc = wave_scan(s);
    const unsigned ex = inc - s;
    reinterpret_cast<uint4*>(sh.tab)[lane] =
        make_uint4(ex, ex + v.x, ex + v.x + v.y, ex + v.x + v.y + v.z);
    if (lane == 63) sh.tab[kNI * kWaves] = inc;
  }
  __syncthreads();
  return sh.tab[kNI * kWaves];
}

// ordered_plan_sparse again, for a new mask, after an earlier plan (or any
// other use of sh.tab) in the same workgroup: the counts are zeroed first.
__device__ inline unsigned replan_sparse(unsigned f, SelShared& sh) {
  if (threadIdx.x < (kNI * kWaves + 4) / 4)
    reinterpret_cast<uint4*>(sh.tab)[threadIdx.x] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  return ordered_plan_sparse(f, sh);
}

template <typename F>
__device__ inline void ordered_apply_sparse(unsigned f, SelShared& sh, F&& fn) {
  const unsigned w = threadIdx.x >> 6;
  for (unsigned any = wave_or(f); any != 0u; any &= any - 1u) {
    const int i = __builtin_ctz(any);
    const unsigned long long b = __ballot((f >> i) & 1u);
    if ((f >> i) & 1u) fn(i, sh.tab[i * kWaves + w] + mbcnt(b));
  }
}

// ---- histograms ------------------------------------------------------------

// hist[bin] += 1 for every lane with act.  The most frequent bin of the wave
// instruction is aggregated with a ballot; the rest use LDS atomics.  Must be
// reached by all lanes of the wave.
__device__ inline void hist_add(unsigned* hist, unsigned bin, bool act) {
  const unsigned long long pend = __ballot(act);
  if (pend == 0) return;
  const int leader = __builtin_ctzll(pend);
  const unsigned b = unsigned(__builtin_amdgcn_readlane(int(bin), leader));
  const unsigned long long same = __ballot(act && bin == b);
  if (lane_id() == unsigned(leader)) atomicAdd(&hist[b], unsigned(__popcll(same)));
  if (act && bin != b) atomicAdd(&hist[bin], 1u);
}

// Number of bits of x (0 for x = 0).
__device__ inline int bit_width(unsigned x) { return x ? 32 - __clz(x) : 0; }

// After a histogram pass: the bin where the running count from the top first
// reaches `need`.  Publishes (digit, need - count above it, bin count).
__device__ inline void find_bin(SelShared& sh, unsigned need) {
  const unsigned t = threadIdx.x, lane = lane_id(), w = t >> 6;
  // thread t holds bins 2047 - 4t .. 2044 - 4t: thread order is descending key
  const uint4 h = reinterpret_cast<const uint4*>(sh.hist)[kThreads - 1 - t];
  const unsigned hb[4] = {h.w, h.z, h.y, h.x};
  const unsigned s = h.x + h.y + h.z + h.w;
  const unsigned inc = wave_scan(s);
  if (lane == 63) sh.red[0][w] = inc;
  __syncthreads();
  unsigned above = inc - s;
#pragma unroll
  for (unsigned w2 = 0; w2 < unsigned(kWaves); ++w2) above += w2 < w ? sh.red[0][w2] : 0u;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (above < need && need <= above + hb[j]) {
      sh.digit = 2047u - 4u * t - unsigned(j);
      sh.need = need - above;
      sh.cnt = hb[j];
    }
    above += hb[j];
  }
  __syncthreads();
}

// ---- bound ------------------------------------------------------------------

// A key that at least `need` of the workgroup's valid keys reach, or 0 when
// there are too few.  The histogram counts maxima of groups of G consecutive
// slots of a lane (distinct candidates, so need maxima reaching a key means
// need candidates do): G = 4 while the 4096 group maxima leave need well
// inside, fewer otherwise; a group counts when its first slot is valid
// (invalid slots hold key 0).  The 2048 bins split [lo, hi] linearly (key -
// lo), so scores that straddle a power of two still spread out; the bound is
// the floor of the bin where the count from the top reaches need.
__device__ inline unsigned group_bound(SelShared& sh, const unsigned (&key)[kNI], unsigned vm,
                                       unsigned need, unsigned G = 0u) {
  // G = 0: choose by need; G = 1 counts every key (e.g. keys that are maxima)
  if (G == 0u) G = need <= 1024u ? 4u : (need <= 2048u ? 2u : 1u);
  unsigned gvm = 0u, gm[kNI], lo = ~0u, hi = 0u;
#pragma unroll
  for (int i = 0; i < kNI; ++i) {
    gm[i] = key[i];
    if (G >= 2u && (i & 1) == 0) gm[i] = max(key[i], key[i + 1]);
    if (G == 4u && (i & 3) == 0) gm[i] = max(max(key[i], key[i + 1]), max(key[i + 2], key[i + 3]));
    if ((unsigned(i) & (G - 1u)) == 0u) gvm |= ((vm >> i) & 1u) << i;
    if ((vm >> i) & 1u) {
      lo = min(lo, key[i]);
      hi = max(hi, key[i]);
    }
  }
  const Red3 r = block_reduce(sh, unsigned(__popc(gvm)), lo, hi);
  if (r.sum < need) return 0u;
  if (r.lo == r.hi) return r.lo;
  const int width = bit_width(r.hi - r.lo);
  const int shift = width > 11 ? width - 11 : 0;  // bins (key - lo) >> shift, all < 2048
  reinterpret_cast<uint4*>(sh.hist)[threadIdx.x] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kNI; ++i)  // groups start at slots i % G == 0 (G is uniform)
    if ((unsigned(i) & (G - 1u)) == 0u) hist_add(sh.hist, (gm[i] - r.lo) >> shift, (gvm >> i) & 1u);
  __syncthreads();
  find_bin(sh, need);
  return r.lo + (sh.digit << shift);
}

// ---- exact cut (fallback) --------------------------------------------------

// Where the top `need` of a set of keys ends: every key > tau is in it, and
// of the keys == tau the first `take` (position order).  take == 0: the cut
// falls on a bin edge and exactly the keys >= tau are in it.
struct Cut {
  unsigned tau, take, ties;
};

// Exact cut for the top need (1 <= need <= valid count) of the workgroup's
// keys.  Radix passes of up to 11 bits run over key - lo (lo: the smallest
// valid key), from its top bit down, and stop early when the boundary bin is
// taken whole.
__device__ inline Cut find_cut(SelShared& sh, const unsigned (&key)[kNI], unsigned vm,
                               unsigned need) {
  unsigned lo = ~0u, hi = 0u;
#pragma unroll
  for (int i = 0; i < kNI; ++i)
    if ((vm >> i) & 1u) {
      lo = min(lo, key[i]);
      hi = max(hi, key[i]);
    }
  const Red3 r = block_reduce(sh, 0u, lo, hi);
  if (r.lo == r.hi) return Cut{r.lo, need, ~0u};  // all equal: ties by position
  int shift = bit_width(r.hi - r.lo);
  unsigned prefix = 0u;  // of key - lo
#pragma nounroll
  for (;;) {
    const int bits = shift < 11 ? shift : 11;
    shift -= bits;
    reinterpret_cast<uint4*>(sh.hist)[threadIdx.x] = make_uint4(0u, 0u, 0u, 0u);
    __syncthreads();
    const unsigned mask = (1u << bits) - 1u;
#pragma unroll
    for (int i = 0; i < kNI; ++i) {
      const unsigned rel = key[i] - r.lo;
      const bool act = ((vm >> i) & 1u) && shr(rel, shift + bits) == prefix;
      hist_add(sh.hist, (rel >> shift) & mask, act);
    }
    __syncthreads();
    find_bin(sh, need);
    prefix = (prefix << bits) | sh.digit;
    need = sh.need;
    const unsigned cnt = sh.cnt;
    if (cnt == need) return Cut{r.lo + (prefix << shift), 0u, 0u};
    if (shift == 0) return Cut{r.lo + prefix, need, cnt};
  }
}

// Selection mask of a cut (bit i: slot i); ties resolved in position order.
__device__ inline unsigned cut_mask(SelShared& sh, const unsigned (&key)[kNI], unsigned vm,
                                    const Cut& c) {
  unsigned ge = 0u, eq = 0u;
#pragma unroll
  for (int i = 0; i < kNI; ++i) {
    ge |= unsigned(c.take == 0u ? key[i] >= c.tau : key[i] > c.tau) << i;
    eq |= unsigned(key[i] == c.tau) << i;
  }
  ge &= vm;
  if (c.take == 0u) return ge;
  eq &= vm;
  if (c.ties > c.take) {
    const Ordered o = ordered_plan(eq, sh);
    unsigned drop = 0u;
    const unsigned take = c.take;
    ordered_apply(eq, o, sh, [&](int i, unsigned rank) { drop |= unsigned(rank >= take) << i; });
    __syncthreads();
    eq &= ~drop;
  }
  return ge | eq;
}

// ---- loads -----------------------------------------------------------------

// Valid-slot mask of a lane for n elements at positions i * kThreads + tid.
__device__ inline unsigned valid_mask(unsigned n) {
  const unsigned t = threadIdx.x;
  const unsigned nv = n > t ? (n - t + kThreads - 1) / kThreads : 0u;
  return nv >= 32u ? ~0u : (1u << nv) - 1u;
}

// Raw scores at chunk positions [base, base + n) of request r.  Invalid slots
// get key 0.  Every lane issues all of its loads before using any (invalid
// slots read a clamped, in-bounds address), so the chunk streams in one
// round trip.
template <bool BEAM>
__device__ inline unsigned load_raw(const SelectParams& p, unsigned r, unsigned base, unsigned n,
                                    unsigned (&key)[kNI]) {
  const unsigned vm = valid_mask(n);
  const float* logp_r = p.logp + size_t(r) * p.N;
  const float* beam_r = BEAM ? p.beam + size_t(r) * p.W_prev : nullptr;
  const unsigned pos0 = base + threadIdx.x;
  float x[kNI], bs[kNI];
  unsigned row = 0u, rem = 0u;  // row of the current position and its offset in the row
  if constexpr (BEAM) {
    const unsigned first = min(pos0, p.N - 1u);
    row = row_of(first, p.V, p.inv_v);
    rem = first - row * p.V;
  }
#pragma unroll
  for (int i = 0; i < kNI; ++i) {
    const bool valid = (vm >> i) & 1u;
    const unsigned pos = pos0 + unsigned(i) * kThreads;
    if constexpr (BEAM) {
      if (i > 0) {
        rem += kThreads;
        if (rem >= p.V) {
          if (p.V >= unsigned(kThreads)) {  // at most one row boundary per step
            rem -= p.V;
            ++row;
          } else {
            row = row_of(valid ? pos : base, p.V, p.inv_v);
            rem = (valid ? pos : base) - row * p.V;
          }
        }
      }
      bs[i] = beam_r[valid ? row : 0u];
    }
    x[i] = logp_r[valid ? pos : base];
  }
#pragma unroll
  for (int i = 0; i < kNI; ++i) {
    float v = x[i];
    if constexpr (BEAM) v = bs[i] + v;
    key[i] = ((vm >> i) & 1u) ? order_key(v) : 0u;
  }
  return vm;
}

// Candidates of the input slots [s0, s0 + group) of request r.  Invalid
// slots get key 0.  Returns the validity mask; sh.scnt holds the counts.
// Loads are unconditional (invalid slots re-read the region's first pair).
__device__ inline unsigned load_slots(const SelectParams& p, SelShared& sh, unsigned r,
                                      unsigned s0, unsigned (&key)[kNI], unsigned (&idx)[kNI]) {
  if (threadIdx.x < p.group) {
    const unsigned s = s0 + threadIdx.x;
    sh.scnt[threadIdx.x] = s < p.nslots_in ? p.cnt_in[size_t(r) * p.nslots_in + s] : 0u;
  }
  __syncthreads();
  const uint2* in = p.cand_in + (size_t(r) * p.nslots_in + s0) * p.cap;
  unsigned vm = 0u;
  uint2 c[kNI];
#pragma unroll
  for (int i = 0; i < kNI; ++i) {
    const unsigned pos = unsigned(i) * kThreads + threadIdx.x;
    const unsigned s = pos >> p.lcap, j = pos & (p.cap - 1u);
    const bool valid = s < p.group && j < sh.scnt[s];
    vm |= unsigned(valid) << i;
    c[i] = in[valid ? pos : 0u];
  }
#pragma unroll
  for (int i = 0; i < kNI; ++i) {
    const bool valid = (vm >> i) & 1u;
    key[i] = valid ? c[i].x : 0u;
    idx[i] = valid ? c[i].y : 0u;
  }
  return vm;
}

// ---- sort ------------------------------------------------------------------

// Stable LSD radix sort of the m (<= kSortCap) composites in a, descending
// by their high 32 bits (the score key), in 8-bit passes over key - lo (lo:
// the smallest key), as many as key - lo needs; the sorted values end in
// the returned buffer (a or b).  The composites arrive in index order and
// every pass is stable, so equal keys stay in index order: the result is the
// (score desc, index asc) order.  Element p of a pass is handled by round p / kThreads, lane p % 64
// of wave (p / 64) % 8; its rank among the equal digits before it is the
// count of lower lanes of its wave with that digit (the digit's lane mask
// from 8 ballots) plus the counts of the earlier (round, wave) pairs.
struct alignas(16) RadixShared {
  union {
    unsigned cnt[kSortCap / kThreads][kWaves][256];
    unsigned flat[kSelectChunk];  // free for other use between sorts
    uint4 flat4[kSelectChunk / 4];
  };
  unsigned tot[256];
};
static_assert(sizeof(unsigned[kSortCap / kThreads][kWaves][256]) == kSelectChunk * sizeof(unsigned),
              "the sort counters span one chunk of words");

__device__ inline unsigned long long* radix_sort_desc(unsigned long long* a, unsigned long long* b,
                                                      unsigned m, unsigned lo, unsigned hi,
                                                      RadixShared& rs) {
  constexpr int RMAX = kSortCap / kThreads;
  const unsigned lane = lane_id(), w = threadIdx.x >> 6;
  const unsigned rounds = (m + kThreads - 1) / kThreads;
  const int passes = (bit_width(hi - lo) + 7) / 8;
  unsigned* cflat = &rs.cnt[0][0][0];
  unsigned long long* src = a;
  unsigned long long* dst = b;
  for (int pass = 0; pass < passes; ++pass) {
    const int shift = 8 * pass;
    for (unsigned i = threadIdx.x; i < rounds * kWaves * 256; i += kThreads) cflat[i] = 0u;
    __syncthreads();
    unsigned long long v[RMAX];
    unsigned dg[RMAX], rk[RMAX];
#pragma unroll
    for (int j = 0; j < RMAX; ++j) {
      if (unsigned(j) < rounds) {
        const unsigned pos = unsigned(j) * kThreads + threadIdx.x;
        const bool valid = pos < m;
        v[j] = valid ? src[pos] : 0ull;
        const unsigned d = 255u - (((unsigned(v[j] >> 32) - lo) >> shift) & 255u);
        unsigned long long same = __ballot(valid);
#pragma unroll
        for (int bit = 0; bit < 8; ++bit) {
          const unsigned long long mb = __ballot((d >> bit) & 1u);
          same &= ((d >> bit) & 1u) ? mb : ~mb;
        }
        rk[j] = mbcnt(same);
        dg[j] = d;
        if (valid && rk[j] == 0u) rs.cnt[j][w][d] = unsigned(__popcll(same));
      }
    }
    __syncthreads();
    if (threadIdx.x < 256) {  // per digit: exclusive prefix over (round, wave)
      const unsigned d = threadIdx.x;
      unsigned run = 0u;
      for (unsigned j = 0; j < rounds; ++j)
        for (int w2 = 0; w2 < kWaves; ++w2) {
          const unsigned c = rs.cnt[j][w2][d];
          rs.cnt[j][w2][d] = run;
          run += c;
        }
      rs.tot[d] = run;
    }
    __syncthreads();
    if (w == 0) {  // exclusive prefix of the digit totals
      const uint4 t4 = reinterpret_cast<const uint4*>(rs.tot)[lane];
      const unsigned sum = t4.x + t4.y + t4.z + t4.w;
      const unsigned ex = wave_scan(sum) - sum;
      reinterpret_cast<uint4*>(rs.tot)[lane] =
          make_uint4(ex, ex + t4.x, ex + t4.x + t4.y, ex + t4.x + t4.y + t4.z);
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < RMAX; ++j) {
      if (unsigned(j) < rounds) {
        const unsigned pos = unsigned(j) * kThreads + threadIdx.x;
        if (pos < m) dst[rs.tot[dg[j]] + rs.cnt[j][w][dg[j]] + rk[j]] = v[j];
      }
    }
    __syncthreads();
    unsigned long long* tmp = src;
    src = dst;
    dst = tmp;
  }
  return src;
}

// ---- kernels ---------------------------------------------------------------

// Superset (or exact set) of the top min(W, n) of one workgroup's candidates
// into slot (r, g): survivors of the bound when they fit, else the exact cut.
template <typename IdxFn>
__device__ inline void reduce_group(const SelectParams& p, SelShared& sh, unsigned r, unsigned g,
                                    const unsigned (&key)[kNI], unsigned vm, unsigned n,
                                    IdxFn&& idx_of) {
  uint2* out = p.cand_out + (size_t(r) * p.nwg + g) * p.cap;
  const unsigned need = min(p.W, n);
  unsigned keep = vm;
  if (n > p.cap) {
    const unsigned b = group_bound(sh, key, vm, need);
#pragma unroll
    for (int i = 0; i < kNI; ++i) keep &= ~(unsigned(key[i] < b) << i);
  }
  Ordered o = ordered_plan(keep, sh);
  if (o.total > p.cap) {
    __syncthreads();
    const Cut c = find_cut(sh, key, vm, need);
    keep = cut_mask(sh, key, vm, c);
    o = ordered_plan(keep, sh);
  }
  ordered_apply(keep, o, sh,
                [&](int i, unsigned rank) { out[rank] = make_uint2(key[i], idx_of(i)); });
  if (threadIdx.x == 0) p.cnt_out[size_t(r) * p.nwg + g] = o.total;
}

template <bool BEAM>
__global__ __launch_bounds__(kThreads) void select_raw_stage_kernel(SelectParams p) {
  __shared__ SelShared sh;
  const unsigned r = blockIdx.x / p.nwg, g = blockIdx.x - r * p.nwg;
  const unsigned base = g * unsigned(kSelectChunk);
  const unsigned n = min(p.N - base, unsigned(kSelectChunk));
  unsigned key[kNI];
  const unsigned vm = load_raw<BEAM>(p, r, base, n, key);
  reduce_group(p, sh, r, g, key, vm, n,
               [&](int i) { return base + unsigned(i) * kThreads + threadIdx.x; });
}

__global__ __launch_bounds__(kThreads) void select_slot_stage_kernel(SelectParams p) {
  __shared__ SelShared sh;
  const unsigned r = blockIdx.x / p.nwg, g = blockIdx.x - r * p.nwg;
  unsigned key[kNI], idx[kNI];
  const unsigned vm = load_slots(p, sh, r, g * p.group, key, idx);
  const Red3 t = block_reduce(sh, unsigned(__popc(vm)), 0u, 0u);
  reduce_group(p, sh, r, g, key, vm, t.sum, [&](int i) { return idx[i]; });
}

// Shared memory of the last stage of a selection.
struct FinalShared {
  SelShared sh;
  unsigned long long srt[kSortCap];
  unsigned long long srt2[kSortCap];
  RadixShared rsh;
};

// Writes the composite c (key, ~index) as pick j of request r: parent beam,
// token and score.
template <bool BEAM>
__device__ inline void emit_pick(const SelectParams& p, unsigned r, unsigned j,
                                 unsigned long long c) {
  const unsigned fi = ~unsigned(c);
  const unsigned key = unsigned(c >> 32);
  const unsigned row = row_of(fi, p.V, p.inv_v);
  const size_t o2 = size_t(r) * p.W + j;
  p.parents[o2] = int(row);
  p.tokens[o2] = int(fi - row * p.V);
  // the key is the score's bit pattern for every number (no re-read); a NaN
  // (key 0) is recomputed so that its own bits come out
  float sc = __uint_as_float((key & 0x80000000u) ? (key & 0x7fffffffu) : ~key);
  if (key == 0u) {
    const float* logp_r = p.logp + size_t(r) * p.N;
    if constexpr (BEAM) sc = p.beam[size_t(r) * p.W_prev + row] + logp_r[fi];
    else sc = logp_r[fi];
  }
  p.scores[o2] = sc;
}

// Sorts the m (key, ~index) pairs in fs.srt (in index order, written before
// the call by any thread) best first and writes the first W to
// parents / tokens / scores of request r.  klo / khi: this thread's share of
// the key range.
template <bool BEAM>
__device__ inline void sort_emit(const SelectParams& p, FinalShared& fs, unsigned r, unsigned m,
                                 unsigned klo, unsigned khi) {
  auto emit = [&](unsigned j, unsigned long long c) { emit_pick<BEAM>(p, r, j, c); };
  __syncthreads();  // srt is written; the caller's reads of fs.sh are done
  const Red3 kr = block_reduce(fs.sh, 0u, klo, khi);
  const unsigned long long* sorted = radix_sort_desc(fs.srt, fs.srt2, m, kr.lo, kr.hi, fs.rsh);
  for (unsigned j = threadIdx.x; j < p.W; j += kThreads) emit(j, sorted[j]);
}

// Top W of the n candidates held in registers (slot i of a lane at position
// i * kThreads + tid, position order = flat-index order), sorted, written to
// parents / tokens / scores of request r.
template <bool BEAM>
__device__ inline void finish_select(const SelectParams& p, FinalShared& fs, unsigned r,
                                     const unsigned (&key)[kNI], const unsigned (&idx)[kNI],
                                     unsigned vm, unsigned n) {
  SelShared& sh = fs.sh;
  unsigned keep = vm;
  if (n > unsigned(kSortCap)) {
    const unsigned b = group_bound(sh, key, vm, p.W);
#pragma unroll
    for (int i = 0; i < kNI; ++i) keep &= ~(unsigned(key[i] < b) << i);
  }
  Ordered o = ordered_plan(keep, sh);
  if (o.total > unsigned(kSortCap)) {
    __syncthreads();
    const Cut c = find_cut(sh, key, vm, p.W);
    keep = cut_mask(sh, key, vm, c);
    o = ordered_plan(keep, sh);
  }
  // Composite: score key high, complemented index low (the index is
  // recovered from it; the sort orders by the key and keeps index order).
  unsigned klo = ~0u, khi = 0u;
#pragma unroll
  for (int i = 0; i < kNI; ++i)
    if ((keep >> i) & 1u) {
      klo = min(klo, key[i]);
      khi = max(khi, key[i]);
    }
  ordered_apply(keep, o, sh, [&](int i, unsigned rank) {
    fs.srt[rank] = (static_cast<unsigned long long>(key[i]) << 32) | unsigned(~idx[i]);
  });
  sort_emit<BEAM>(p, fs, r, o.total, klo, khi);
}

// Top W of request r's last candidates, sorted, into parents/tokens/scores.
template <bool RAW, bool BEAM>
__global__ __launch_bounds__(kThreads) void select_final_kernel(SelectParams p) {
  __shared__ FinalShared fs;
  const unsigned r = blockIdx.x;
  unsigned key[kNI], idx[kNI], vm, n;
  if constexpr (RAW) {
    n = p.N;
    vm = load_raw<BEAM>(p, r, 0u, n, key);
#pragma unroll
    for (int i = 0; i < kNI; ++i) idx[i] = unsigned(i) * kThreads + threadIdx.x;
  } else {
    vm = load_slots(p, fs.sh, r, 0u, key, idx);
    n = block_reduce(fs.sh, unsigned(__popc(vm)), 0u, 0u).sum;
  }
  finish_select<BEAM>(p, fs, r, key, idx, vm, n);
}

// ---- two-pass path ----------------------------------------------------------
// For W_prev * V >= 2 W * 2048 (and at most 16384 * 2048) candidates:
//   segmax: every wave of a raw chunk writes the largest key of its 2048
//     candidates;
//   filter: every workgroup takes as bound a key that at least W of the
//     request's wave maxima reach (one histogram pass over them) -- W maxima
//     are W distinct candidates, so no member of the top W is below it --
//     re-reads its chunk and keeps the candidates at or above the bound, in
//     index order, in its chunk's slot of `cap` (>= W) pairs, with the count
//     and the chunk's largest key; a chunk with more survivors than the slot
//     holds keeps their exact top W;
//   place (at most kThreads chunks and W <= kOnePassRankMax): the filter's
//     slots and counts have the one-pass layout, and the one-pass path's
//     placing kernel finishes the call exactly as it finishes that path;
//   rank (more chunks): up to kRankCap survivors (the usual case), workgroups
//     of the whole chip each load every survivor of the request into LDS and
//     rank 32 of them: a survivor's place in the result is the number of survivors
//     before it in the total order (composite (key, ~index) compared as one
//     64-bit integer, unique per candidate), and those placed below W are
//     written out directly: no sort and no single-workgroup pass;
//   gather (more survivors): one workgroup per request walks the slots in
//     chunk order (index order), 16384 candidates at a time, keeping the
//     exact top W of what it has seen in LDS between rounds, and finishes
//     like the final kernel.  Every later candidate has a higher index than
//     the kept ones, so once W are kept it can only enter with a key above
//     their smallest: slots whose largest key is not above it are skipped
//     whole, and so are such candidates.
// For smooth score distributions about W candidates survive the bound.

template <bool BEAM>
__global__ __launch_bounds__(kThreads) void select_segmax_kernel(SelectParams p) {
  const unsigned r = blockIdx.x / p.nwg, c = blockIdx.x - r * p.nwg;
  const unsigned base = c * unsigned(kSelectChunk);
  const unsigned n = min(p.N - base, unsigned(kSelectChunk));
  unsigned key[kNI];
  load_raw<BEAM>(p, r, base, n, key);
  unsigned mx = 0u;
#pragma unroll
  for (int i = 0; i < kNI; ++i) mx = max(mx, key[i]);  // invalid slots hold 0
  const Red3 w = wave_reduce(0u, 0u, mx);
  if (lane_id() == 0) p.segmax[size_t(r) * p.nseg + c * kWaves + (threadIdx.x >> 6)] = w.hi;
}

template <bool BEAM, bool WORD>
__global__ __launch_bounds__(kThreads) void select_filter_kernel(SelectParams p) {
  __shared__ SelShared sh;
  const unsigned r = blockIdx.x / p.nwg, c = blockIdx.x - r * p.nwg;
  const unsigned base = c * unsigned(kSelectChunk);
  const unsigned n = min(p.N - base, unsigned(kSelectChunk));
  unsigned key[kNI];
  const unsigned vm = load_raw<BEAM>(p, r, base, n, key);
  unsigned bound;
  if constexpr (WORD) {
    // the request's bound word, formed in the summary pass as the one-pass
    // path forms it: keys below B are dropped, and keys equal to B beyond c*
    const unsigned long long bw = p.tp_bound[r];
    const unsigned B = unsigned(bw), cstar = unsigned(bw >> 32) - 1u;
    bound = (c > cstar && B < ~0u) ? B + 1u : B;
  } else {
    // wave maxima of the request; segment (chunk s / 8, wave s % 8) exists
    // when its first candidate does
    // (only the rows i * kThreads < nseg are read: a workgroup-uniform
    // bound, so no load is issued for the empty tail of the lanes' slots)
    unsigned mk[kNI], mvm = 0u;
    const unsigned* seg = p.segmax + size_t(r) * p.nseg;
#pragma unroll
    for (int i = 0; i < kNI; ++i) {
      mk[i] = 0u;
      if (unsigned(i) * kThreads < p.nseg) {
        const unsigned s = unsigned(i) * kThreads + threadIdx.x;
        const bool valid =
            s < p.nseg && (s / kWaves) * unsigned(kSelectChunk) + (s % kWaves) * 64u < p.N;
        mk[i] = seg[valid ? s : 0u];
        mvm |= unsigned(valid) << i;
      }
    }
#pragma unroll
    for (int i = 0; i < kNI; ++i) mk[i] = ((mvm >> i) & 1u) ? mk[i] : 0u;
    // at least W maxima reach the bound (floor of the histogram bin where
    // their count from the top reaches W)
    bound = group_bound(sh, mk, mvm, p.W, 1u);
  }
  unsigned keep = vm;
#pragma unroll
  for (int i = 0; i < kNI; ++i) keep &= ~(unsigned(key[i] < bound) << i);
  if (threadIdx.x < (kNI * kWaves + 4) / 4)  // the sparse compaction's zero counts
    reinterpret_cast<uint4*>(sh.tab)[threadIdx.x] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  uint2* out = p.cand_out + (size_t(r) * p.nwg + c) * p.cap;
  auto put = [&](int i, unsigned rank) {
    out[rank] = make_uint2(key[i], base + unsigned(i) * kThreads + threadIdx.x);
  };
  unsigned total = ordered_plan_sparse(keep, sh);
  if (total > p.cap) {  // rare: keep the chunk's exact top W of the survivors
    __syncthreads();
    keep = cut_mask(sh, key, keep, find_cut(sh, key, keep, p.W));
    total = replan_sparse(keep, sh);
    ordered_apply_sparse(keep, sh, put);
  } else {
    ordered_apply_sparse(keep, sh, put);
  }
  if (threadIdx.x == 0) {  // (count, largest key of the chunk: its waves' maxima)
    unsigned top = 0u;
    const size_t s0 = size_t(r) * p.nseg + c * kWaves;
    for (int w = 0; w < kWaves; ++w)
      top = max(top, WORD ? p.ex[s0 + unsigned(w)].x : p.segmax[s0 + unsigned(w)]);
    reinterpret_cast<uint2*>(p.cnt_out)[size_t(r) * p.nwg + c] = make_uint2(total, top);
  }
}

// Inclusive running maximum over the 64 lanes.
__device__ inline unsigned wave_scan_max(unsigned x) {
  x = max(x, dppu<0x111>(x));       // row_shr:1
  x = max(x, dppu<0x112>(x));       // row_shr:2
  x = max(x, dppu<0x114>(x));       // row_shr:4
  x = max(x, dppu<0x118>(x));       // row_shr:8
  x = max(x, dppu<0x142, 0xA>(x));  // row_bcast:15 into rows 1, 3
  x = max(x, dppu<0x143, 0xC>(x));  // row_bcast:31 into rows 2, 3
  return x;
}

// The multi-round gather of request r (fs, next: the workgroup's LDS;
// next[] holds the (slot, offset) where the next round starts).
template <bool BEAM>
__device__ inline void gather_rounds(const SelectParams& p, FinalShared& fs, unsigned (&next)[2],
                                     unsigned r) {
  // Round position q -> 1 + (index of its pair in the request's slots) - q,
  // in fs.rsh.flat (the radix sort's counters are idle until the last
  // round).  Within a live slot that difference is constant, and it does not
  // decrease from slot to slot (a slot holds at most cap pairs), so writing
  // it at each slot's first position and taking a running maximum fills the
  // map.
  const unsigned ns = p.nslots_in;
  const unsigned lane = lane_id(), w = threadIdx.x >> 6;
  const uint2* slots = p.cand_in + size_t(r) * ns * p.cap;
  unsigned c4[4], m4[4];  // count and largest key of slots 4t .. 4t + 3 (ns <= 4 * kThreads)
  {
    const uint2* cm = reinterpret_cast<const uint2*>(p.cnt_in) + size_t(r) * ns;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const unsigned sl = 4u * threadIdx.x + unsigned(q);
      const uint2 e = cm[sl < ns ? sl : 0u];
      c4[q] = sl < ns ? e.x : 0u;
      m4[q] = e.y;
    }
  }
  unsigned cur = 0u, off = 0u, carried = 0u, floor_key = 0u;
  for (;;) {
    // The thread id is re-read every round so that the compiler rebuilds the
    // per-slot positions here instead of keeping 32 of them live across rounds.
    unsigned t = threadIdx.x;
    asm volatile("" : "+v"(t));
    // live counts: slots before cur are consumed, cur up to off; with W kept,
    // a slot whose largest key does not beat the smallest kept one is dead
    unsigned v[4], sum = 0u;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const unsigned sl = 4u * t + unsigned(q);
      unsigned c = sl < cur ? 0u : c4[q] - (sl == cur ? off : 0u);
      if (carried > 0u && m4[q] <= floor_key) c = 0u;
      v[q] = c;
      sum += c;
    }
#pragma unroll
    for (int i = 0; i < kNI; ++i) fs.rsh.flat[unsigned(i) * kThreads + t] = 0u;
    const unsigned inc = wave_scan(sum);
    if (lane == 63) fs.sh.red[0][w] = inc;
    __syncthreads();
    unsigned run = inc - sum, total = 0u;
#pragma unroll
    for (int w2 = 0; w2 < kWaves; ++w2) {
      const unsigned x = fs.sh.red[0][w2];
      total += x;
      run += unsigned(w2) < w ? x : 0u;
    }
    const unsigned room = unsigned(kSelectChunk) - carried;
    const unsigned fresh = total < room ? total : room;
    const bool last = fresh == total;
    unsigned st[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const unsigned sl = 4u * t + unsigned(q);
      st[q] = run;
      // live slots start at distinct positions; sl * cap + skipped >= run
      if (v[q] > 0u && run < fresh)
        fs.rsh.flat[run] = 1u + (sl << p.lcap) + (sl == cur ? off : 0u) - run;
      run += v[q];
    }
    __syncthreads();
    {  // running maximum over the map: thread t holds entries 32t .. 32t + 31
      uint4 a[8];
      unsigned mx = 0u;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        a[k] = fs.rsh.flat4[8u * t + unsigned(k)];
        mx = max(mx, max(max(a[k].x, a[k].y), max(a[k].z, a[k].w)));
      }
      const unsigned wi = wave_scan_max(mx);
      if (lane == 63) fs.sh.red[1][w] = wi;
      // exclusive across lanes: lane - 1's inclusive value
      unsigned pre = unsigned(__shfl_up(int(wi), 1));
      if (lane == 0) pre = 0u;
      __syncthreads();
#pragma unroll
      for (int w2 = 0; w2 < kWaves; ++w2) pre = unsigned(w2) < w ? max(pre, fs.sh.red[1][w2]) : pre;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        a[k].x = pre = max(pre, a[k].x);
        a[k].y = pre = max(pre, a[k].y);
        a[k].z = pre = max(pre, a[k].z);
        a[k].w = pre = max(pre, a[k].w);
        fs.rsh.flat4[8u * t + unsigned(k)] = a[k];
      }
    }
    __syncthreads();
    if (carried == 0u && total <= unsigned(kSortCap)) {
      // every survivor fits the sort: straight from the slots into it
      unsigned long long pr[kSortCap / kThreads];
      unsigned klo = ~0u, khi = 0u;
#pragma unroll
      for (int i = 0; i < kSortCap / kThreads; ++i) {
        const unsigned q = unsigned(i) * kThreads + t;
        const bool ok = q < total;
        const unsigned d = fs.rsh.flat[ok ? q : 0u];
        const unsigned at = ok ? q + d - 1u : 0u;
        const uint2 e = *reinterpret_cast<const uint2*>(reinterpret_cast<const char*>(slots) +
                                                        at * unsigned(sizeof(uint2)));
        pr[i] = (static_cast<unsigned long long>(e.x) << 32) | unsigned(~e.y);
        klo = ok ? min(klo, e.x) : klo;
        khi = ok ? max(khi, e.x) : khi;
      }
      __syncthreads();  // the map has been read (it shares storage with the sort)
#pragma unroll
      for (int i = 0; i < kSortCap / kThreads; ++i) {
        const unsigned q = unsigned(i) * kThreads + t;
        if (q < total) fs.srt[q] = pr[i];
      }
      sort_emit<BEAM>(p, fs, r, total, klo, khi);
      return;
    }
    // candidates: the carry (positions < carried, from LDS) then `fresh` from
    // the slots; every load is issued unconditionally from a clamped address
    unsigned key[kNI], idx[kNI], fm = 0u;
#pragma unroll
    for (int i = 0; i < kNI; ++i) {
      const unsigned j = unsigned(i) * kThreads + t;
      const unsigned q = j - carried;
      const bool in_fresh = j >= carried && q < fresh;
      const unsigned d = fs.rsh.flat[in_fresh ? q : 0u];
      const unsigned at = in_fresh ? q + d - 1u : 0u;  // pair index, < 2048 * 4096
      const uint2 e = *reinterpret_cast<const uint2*>(reinterpret_cast<const char*>(slots) +
                                                      at * unsigned(sizeof(uint2)));
      key[i] = e.x;
      idx[i] = e.y;
      fm |= unsigned(in_fresh) << i;
    }
    unsigned vm = 0u;
#pragma unroll
    for (int i = 0; i < kNI; ++i) {
      const bool ok = ((fm >> i) & 1u) && !(carried > 0u && key[i] <= floor_key);
      vm |= unsigned(ok) << i;
      key[i] = ok ? key[i] : 0u;
    }
#pragma unroll
    for (int i = 0; i < kSortCap / kThreads; ++i) {  // the carry: positions < carried <= W
      const unsigned j = unsigned(i) * kThreads + t;
      if (j < carried) {
        const unsigned long long cv = fs.srt2[j];
        key[i] = unsigned(cv >> 32);
        idx[i] = ~unsigned(cv);
        vm |= 1u << i;
      }
    }
    __syncthreads();  // the carry and the map have been read
    if (!last) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (v[q] > 0u && st[q] <= fresh && fresh < st[q] + v[q]) {
          const unsigned sl = 4u * t + unsigned(q);
          next[0] = sl;
          next[1] = (sl == cur ? off : 0u) + (fresh - st[q]);
        }
    }
    const unsigned live = block_reduce(fs.sh, unsigned(__popc(vm)), 0u, 0u).sum;
    if (last) {
      finish_select<BEAM>(p, fs, r, key, idx, vm, live);
      return;
    }
    cur = next[0];
    off = next[1];
    if (live == carried) continue;  // nothing fresh beats the carry
    // keep the exact top W seen so far (in index order)
    const Cut cut = find_cut(fs.sh, key, vm, p.W);
    const unsigned keep = cut_mask(fs.sh, key, vm, cut);
    const Ordered o = ordered_plan(keep, fs.sh);
    unsigned kmin = ~0u;
    ordered_apply(keep, o, fs.sh, [&](int i, unsigned rank) {
      fs.srt2[rank] = (static_cast<unsigned long long>(key[i]) << 32) | unsigned(~idx[i]);
      kmin = min(kmin, key[i]);
    });
    floor_key = block_reduce(fs.sh, 0u, kmin, 0u).lo;
    carried = o.total;
  }
}

// LDS of the rank kernel's usual path.
struct RankShared {
  unsigned start[kSelectMaxGatherSlots + 1];  // slot s holds positions [start[s], start[s+1])
  alignas(16) unsigned long long all[kRankCap + 128];  // every survivor's composite, by position
  unsigned red[kWaves];                                 // (+ what the counting loop overreads)
};

template <bool BEAM>
__global__ __launch_bounds__(kThreads) void select_rank_kernel(SelectParams p) {
  __shared__ union {
    RankShared rk;
    FinalShared fs;
  } u;
  __shared__ unsigned next[2];
  const unsigned r = blockIdx.x / kRankBlocks, b = blockIdx.x - r * kRankBlocks;
  const unsigned ns = p.nslots_in, t = threadIdx.x;
  const unsigned lane = lane_id(), w = t >> 6;
  // slot counts (thread t: slots 4t .. 4t + 3) and their exclusive prefix
  unsigned c4[4], sum = 0u;
  {  // (slots beyond ns read as zero counts, without a branch)
    const __amdgpu_buffer_rsrc_t rs =
        buffer_rsrc(reinterpret_cast<const uint2*>(p.cnt_in) + size_t(r) * ns, int(ns * 8u));
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      c4[q] = __builtin_amdgcn_raw_buffer_load_b32(rs, (4u * t + unsigned(q)) * 8u, 0, 0);
      sum += c4[q];
    }
  }
  const unsigned inc = wave_scan(sum);
  if (lane == 63) u.rk.red[w] = inc;
  __syncthreads();
  unsigned run = inc - sum, total = 0u;
#pragma unroll
  for (int w2 = 0; w2 < kWaves; ++w2) {
    const unsigned x = u.rk.red[w2];
    total += x;
    run += unsigned(w2) < w ? x : 0u;
  }
  if (total > unsigned(kRankCap)) {  // rare: the multi-round gather, one workgroup
    if (b == 0) {
      __syncthreads();  // u.rk has been read
      gather_rounds<BEAM>(p, u.fs, next, r);
    }
    return;
  }
  if (b * unsigned(kRankPer) >= total) return;  // nothing of this request to rank here
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const unsigned sl = 4u * t + unsigned(q);
    if (sl < ns) u.rk.start[sl] = run;
    run += c4[q];
  }
  if (t == 0) u.rk.start[ns] = total;
  __syncthreads();
  // every survivor into LDS: position q lies in the last slot whose start is
  // <= q (empty slots share the next one's start, which is then > q)
  const uint2* slots = p.cand_in + size_t(r) * ns * p.cap;
  for (unsigned q = t; q < total; q += kThreads) {
    unsigned lo = 0u, hi = ns;  // start[lo] <= q < start[hi]
    while (hi - lo > 1u) {
      const unsigned mid = (lo + hi) >> 1;
      if (u.rk.start[mid] <= q) lo = mid;
      else hi = mid;
    }
    const uint2 e = slots[size_t(lo) * p.cap + (q - u.rk.start[lo])];
    u.rk.all[q] = (static_cast<unsigned long long>(e.x) << 32) | unsigned(~e.y);
  }
  __syncthreads();
  // survivor i = 32 b + t / 16: its rank is the number of larger composites,
  // counted by 16 lanes over interleaved pairs of positions, four pairs per
  // lane in flight (positions up to total + 127 < kRankCap + 128 are read;
  // the ones at or beyond total are not counted)
  const unsigned i = b * unsigned(kRankPer) + (t >> 4), sub = t & 15u;
  const unsigned long long mine = u.rk.all[i < total ? i : 0u];
  unsigned cnt = 0u;
  for (unsigned j0 = 0; j0 < total; j0 += 128u) {
    ulonglong2 x[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      x[k] = *reinterpret_cast<const ulonglong2*>(&u.rk.all[j0 + 32u * unsigned(k) + 2u * sub]);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const unsigned j = j0 + 32u * unsigned(k) + 2u * sub;
      cnt += unsigned(j < total && x[k].x > mine) + unsigned(j + 1u < total && x[k].y > mine);
    }
  }
  cnt += dppu<0xB1>(cnt);   // quad_perm [1,0,3,2]
  cnt += dppu<0x4E>(cnt);   // quad_perm [2,3,0,1]
  cnt += dppu<0x141>(cnt);  // row_half_mirror
  cnt += dppu<0x140>(cnt);  // row_mirror
  if (sub == 0u && i < total && cnt < p.W) emit_pick<BEAM>(p, r, cnt, mine);
}

// ---- one-pass path ---------------------------------------------------------
// The two-pass path reads every score twice (wave maxima, then the filter).
// When all R * nchunks workgroups of a call can be resident at once (and
// R <= kSelectOnePassMaxRequests, W <= kOnePassRankMax), one pass over the
// scores does the filtering, each chunk held in registers from its single
// read, and a small second launch places the survivors:
//   1. every wave publishes (M, m, kM): its largest key M, the smallest of
//      its live lanes' largest keys m, and the number kM of lanes whose
//      largest key is M.  Each lane's largest key is a distinct candidate,
//      so the wave guarantees kM candidates at keys <= M and all its nl live
//      lanes' candidates at keys <= m.  The summary carries the call's tag;
//   2. the request's first workgroup reads the wave summaries until all of
//      them carry the tag (no counter: it sees the last one about one load
//      round trip after it lands, with every summary already loaded) and takes
//      as bound B a key at which the guaranteed count reaches W, so that no
//      member of the top W lies below it: the floor of the bin where the
//      count from the top reaches W after two 11-bit histogram passes (to
//      2^-22 of the key range), raised to the next summary key.  It also finds the first chunk c* at which
//      the chunks' guaranteed counts at B, summed in index order, reach W:
//      a candidate of a later chunk whose key equals B has W better ones
//      (equal or higher keys at lower indices), so it cannot be kept (this
//      keeps tied scores from surviving in every chunk).  B is published
//      before c*, for which only chunks holding a key equal to B wait.  The
//      others wait for the bound word for a bounded time; one that gives up
//      keeps its chunk's exact top W instead (slower, never wrong);
//   3. every workgroup keeps its candidates above B, or equal to B in a
//      chunk up to c*, in its chunk's slot, in index order (the chunk's
//      exact top W when they overflow it), with the count and the chunk's
//      largest key;
//   4. the final kernel places the survivors: each one's place is the number
//      of larger (key, ~index) composites, counted directly (up to
//      kBruteRankMax survivors) or through a key histogram (up to kRankCap;
//      staged in LDS by each of the request's fparts workgroups, which place
//      a share each); with more,
//      one workgroup finds their exact top W first (radix cut, ties in index
//      order, re-reading the slots on every pass).  It also returns the
//      request's bound word to zero and advances the epoch.
// The lane-level summaries make the bound tight also when the scores rise
// with the beam (the top W all in the last rows): wave maxima alone then
// guarantee only one candidate per wave.

// The bound word of a request: (h << 32) | B.  h = 0: nothing yet; h =
// kCstarPending: B is known and c* is not; otherwise h = c* + 1.  A call
// that gave up on the summaries publishes B = 0 with h = kNoBound (no chunk
// above c*, so nothing is dropped).
constexpr unsigned kCstarPending = ~0u;
constexpr unsigned kNoBound = ~0u - 1u;

// Waits (thread 0) for the bound word of a request, for B alone or (final)
// also for c*; 0 after `ticks`.
__device__ inline unsigned long long wait_bound(unsigned long long* word,
                                                unsigned long long ticks, bool final) {
  const unsigned long long t0 = static_cast<unsigned long long>(wall_clock64());
  for (;;) {
    const unsigned long long v = __hip_atomic_load(word, __ATOMIC_RELAXED,
                                                   __HIP_MEMORY_SCOPE_AGENT);
    const unsigned h = unsigned(v >> 32);
    if (h != 0u && !(final && h == kCstarPending)) return v;
    if (static_cast<unsigned long long>(wall_clock64()) - t0 > ticks) return 0ull;
    __builtin_amdgcn_s_sleep(2);
  }
}

// Data that crosses workgroups of one pass launch (the XCDs' L2 caches are
// not coherent with each other) is written and read at agent scope (cache
// policy sc1, as the compiler emits for agent-scope atomics): such stores
// write through to memory and such loads bypass the compute unit's and the
// XCD's caches, so no cache-wide write-back or invalidation (an agent-scope
// fence, several microseconds with 256 workgroups issuing them) is needed.
constexpr int kAgentScope = 16;  // cache policy bit sc1
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
__device__ inline void st_agent4(void* base, unsigned off, uint4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), buffer_rsrc(base), off, 0,
                                         kAgentScope);
}
__device__ inline uint4 ld_agent4(__amdgpu_buffer_rsrc_t rs, unsigned off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, kAgentScope));
}
// Waits for this wave's stores to complete (the vector memory counter also
// covers stores on this architecture), before a counter tells others that
// they are there.
__device__ inline void wait_stores() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

// Tags of the one-pass wave summaries.  A summary (M, m, kM) is stored as one
// 16-byte word whose last field is tag ^ mix(M, m, kM), tag = epoch + 1 of the
// call that wrote it; a summary is current when its last field gives back the
// current call's tag.  Every tag a summary in the region carries is at most
// the current epoch (each one-pass call writes epoch + 1, and its final kernel
// then advances the epoch to that value), so only this call's summaries match;
// the region's zero fill reads as tag 0, which no call uses.  The mix (zero
// at zero) makes a read that mixed fields of two different stores fail the
// test as well, without relying on 16-byte stores being seen whole.
__device__ inline unsigned summary_mix(unsigned M, unsigned m, unsigned km) {
  return (M * 0x9E3779B1u) ^ __builtin_rotateleft32(m * 0x85EBCA77u, 13) ^ (km * 0xC2B2AE3Du);
}
__device__ inline unsigned summary_tag(uint4 e) { return e.w ^ summary_mix(e.x, e.y, e.z); }

// Live lanes of wave w of chunk c (lanes holding at least one candidate).
__device__ inline unsigned wave_live_lanes(const SelectParams& p, unsigned c, unsigned w) {
  const unsigned nc = min(p.N - c * unsigned(kSelectChunk), unsigned(kSelectChunk));
  const unsigned first = 64u * w;
  return nc > first ? min(nc - first, 64u) : 0u;
}

// LDS of the bound (the request's first workgroup only).
constexpr int kBoundList = 512;  // events of one histogram bin resolved by brute force
struct BoundShared {
  uint2 ev[kBoundList];          // (key, weight) of the events in the chosen bin
  unsigned nev;
  unsigned red[2][kWaves];
  unsigned late[kWaves];         // threads of each wave whose poll gave up
  alignas(16) unsigned gc[kOnePassSegPer * kThreads / kWaves];  // guaranteed count at B per chunk
};

// Reads request r's wave summaries until every one of this thread's carries
// `tag` (thread t: summaries i * kThreads + t, all rows loaded in each round,
// the ones beyond nseg outside the buffer, reading zeros); 1 when the waiting
// time passed first.  No barrier: onepass_bound's first one joins the threads.
__device__ inline int onepass_poll(const SelectParams& p, unsigned r, unsigned tag,
                                   uint4 (&e)[kOnePassSegPer]) {
  const unsigned nseg = p.nseg, t = threadIdx.x;
  const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(p.ex + size_t(r) * nseg, int(nseg * 16u));
  unsigned pending = 0u;
#pragma unroll
  for (int i = 0; i < kOnePassSegPer; ++i)
    pending |= unsigned(unsigned(i) * kThreads + t < nseg) << i;
  const unsigned long long t0 = static_cast<unsigned long long>(wall_clock64());
  int late = 0;
  while (pending != 0u) {
#pragma unroll
    for (int i = 0; i < kOnePassSegPer; ++i) e[i] = ld_agent4(rs, (unsigned(i) * kThreads + t) * 16u);
#pragma unroll
    for (int i = 0; i < kOnePassSegPer; ++i)
      if (summary_tag(e[i]) == tag) pending &= ~(1u << i);
    if (static_cast<unsigned long long>(wall_clock64()) - t0 > p.wait_ticks) {
      late = 1;
      break;
    }
  }
  return late;
}

// Bound word of request r from every wave's summary (see step 2 above):
// ((c* + 1) << 32) | B, also published to `word` (thread 0): first with B
// alone, then with c*.  Thread t holds summaries i * kThreads + t in e[i]
// (nseg <= kOnePassSegPer * kThreads) from onepass_poll, which gave up when
// `late` is set in any thread: then the word says no bound (B = 0).
//
// Each live summary (M, m, kM) of a wave with nl live lanes is two weighted
// events: (M, kM) and (m, nl - kM).  The guaranteed count at a key x is the
// total weight of the events at keys >= x (for m >= x: kM + nl - kM = nl;
// for M >= x > m: kM), so B, the largest key whose guaranteed count reaches
// W, is the key of the event at which the weight counted from the top
// reaches W.  A 2048-bin weight histogram over key - lo finds the bin that
// holds it; the events of that bin (usually a few) are then compared with
// each other directly.  A bin with more than kBoundList events is split by a
// second histogram pass over the next 11 bits; should that one hold too many
// as well, B is its smallest event key (its count still reaches W).
template <int ROWS = kOnePassSegPer>
__device__ inline unsigned long long onepass_bound(const SelectParams& p, SelShared& sh,
                                                   BoundShared& bs, const uint4 (&e)[ROWS],
                                                   int late, unsigned long long* word) {
  const unsigned nseg = p.nwg * unsigned(kWaves);
  const unsigned t = threadIdx.x, lane = lane_id(), w = t >> 6;
  const unsigned W = p.W;
  reinterpret_cast<uint4*>(sh.hist)[t] = make_uint4(0u, 0u, 0u, 0u);
  if (t == 0) bs.nev = 0u;
  unsigned nl[ROWS], lo = ~0u, hi = 0u;
#pragma unroll
  for (int i = 0; i < ROWS; ++i) {
    nl[i] = 0u;
    if (unsigned(i) * kThreads < nseg) {
      const unsigned s = unsigned(i) * kThreads + t;
      nl[i] = s < nseg ? wave_live_lanes(p, s / kWaves, s % kWaves) : 0u;
      if (nl[i] > 0u) {
        lo = min(lo, e[i].y);
        hi = max(hi, e[i].x);
      }
    }
  }
  {  // (with the poll's wait flags: one barrier for both)
    const Red3 wr = wave_reduce(unsigned(late), lo, hi);
    if (lane == 0) {
      bs.red[0][w] = wr.lo;
      bs.red[1][w] = wr.hi;
      bs.late[w] = wr.sum;
    }
  }
  __syncthreads();
  lo = ~0u;
  hi = 0u;
  unsigned nlate = 0u;
#pragma unroll
  for (int w2 = 0; w2 < kWaves; ++w2) {
    lo = min(lo, bs.red[0][w2]);
    hi = max(hi, bs.red[1][w2]);
    nlate += bs.late[w2];
  }
  if (nlate != 0u) {
    const unsigned long long none = static_cast<unsigned long long>(kNoBound) << 32;
    if (t == 0) __hip_atomic_store(word, none, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return none;
  }
  unsigned B = lo;
  if (lo < hi) {
    int shift = bit_width(hi - lo);
    unsigned prefix = 0u, need = W;
    bool done = false;
    for (int pass = 0; pass < 2 && !done; ++pass) {  // workgroup-uniform
      const int bits = shift < 11 ? shift : 11;
      shift -= bits;
      const unsigned mask = (1u << bits) - 1u;
      if (pass > 0) {
        reinterpret_cast<uint4*>(sh.hist)[t] = make_uint4(0u, 0u, 0u, 0u);
        if (t == 0) bs.nev = 0u;
        __syncthreads();
      }
      // weights by bin, among the events inside the bin chosen so far
#pragma unroll
      for (int i = 0; i < ROWS; ++i)
        if (nl[i] > 0u) {
          const unsigned rm = e[i].x - lo, rl = e[i].y - lo;
          if (shr(rm, shift + bits) == prefix) atomicAdd(&sh.hist[(rm >> shift) & mask], e[i].z);
          if (nl[i] > e[i].z && shr(rl, shift + bits) == prefix)
            atomicAdd(&sh.hist[(rl >> shift) & mask], nl[i] - e[i].z);
        }
      __syncthreads();
      find_bin(sh, need);  // the live lanes (>= N / 32 >= W) always reach W
      prefix = (prefix << bits) | sh.digit;
      need = sh.need;
      // the events of the chosen bin
#pragma unroll
      for (int i = 0; i < ROWS; ++i)
        if (nl[i] > 0u) {
          const unsigned rm = e[i].x - lo, rl = e[i].y - lo;
          if (shr(rm, shift) == prefix) {
            const unsigned q = atomicAdd(&bs.nev, 1u);
            if (q < unsigned(kBoundList)) bs.ev[q] = make_uint2(e[i].x, e[i].z);
          }
          if (nl[i] > e[i].z && shr(rl, shift) == prefix) {
            const unsigned q = atomicAdd(&bs.nev, 1u);
            if (q < unsigned(kBoundList)) bs.ev[q] = make_uint2(e[i].y, nl[i] - e[i].z);
          }
        }
      __syncthreads();
      const unsigned n = bs.nev;
      if (n <= unsigned(kBoundList)) {
        // B = the largest event key x of the bin whose weight at keys >= x,
        // within the bin, reaches need (the bin's smallest key always does)
        unsigned cand = 0u;
        if (t < n) {
          const unsigned x = bs.ev[t].x;
          unsigned g = 0u;
          for (unsigned u = 0; u < n; ++u) {
            const uint2 o = bs.ev[u];
            g += o.x >= x ? o.y : 0u;
          }
          cand = g >= need ? x : 0u;
        }
        const Red3 wr = wave_reduce(0u, 0u, cand);
        if (lane == 0) bs.red[1][w] = wr.hi;
        __syncthreads();
        B = 0u;
#pragma unroll
        for (int w2 = 0; w2 < kWaves; ++w2) B = max(B, bs.red[1][w2]);
        done = true;
      }
    }
    if (!done) {
      // still too many events in the bin: its smallest event key
      const unsigned floor = lo + (prefix << shift);
      unsigned nb = ~0u;
#pragma unroll
      for (int i = 0; i < ROWS; ++i)
        if (nl[i] > 0u) {
          if (e[i].x >= floor) nb = min(nb, e[i].x);
          if (nl[i] > e[i].z && e[i].y >= floor) nb = min(nb, e[i].y);
        }
      const Red3 wr = wave_reduce(0u, nb, 0u);
      if (lane == 0) bs.red[0][w] = wr.lo;
      __syncthreads();
      B = ~0u;
#pragma unroll
      for (int w2 = 0; w2 < kWaves; ++w2) B = min(B, bs.red[0][w2]);
    }
  }
  // B alone first: only chunks holding a key equal to B wait for c*
  if (t == 0)
    __hip_atomic_store(word, (static_cast<unsigned long long>(kCstarPending) << 32) | B,
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // c*: the chunks' guaranteed counts at B, summed in chunk order.  Thread t
  // holds summary i * kThreads + t, i.e. wave t % 8 of chunk i * 64 + t / 8:
  // a chunk's count is a sum over 8 adjacent lanes, stored by the first of
  // them (rows beyond nseg have no live lanes and store zeros); one wave
  // then scans the chunks in order.
#pragma unroll
  for (int i = 0; i < ROWS; ++i) {
    unsigned g = nl[i] > 0u ? (e[i].y >= B ? nl[i] : (e[i].x >= B ? e[i].z : 0u)) : 0u;
    g += dppu<0xB1>(g);   // quad_perm [1,0,3,2]
    g += dppu<0x4E>(g);   // quad_perm [2,3,0,1]
    g += dppu<0x141>(g);  // row_half_mirror: the other quad of the 8 lanes
    if ((lane & 7u) == 0u) bs.gc[unsigned(i) * 64u + t / 8u] = g;
  }
#pragma unroll
  for (int i = ROWS; i < kOnePassSegPer; ++i)  // chunks beyond the rows held: none
    if ((lane & 7u) == 0u) bs.gc[unsigned(i) * 64u + t / 8u] = 0u;
  if (t == 0) sh.digit = ~0u;  // (c* always exists: the counts at B reach W)
  __syncthreads();
  if (w == 0) {  // lane l: chunks 8 l .. 8 l + 7
    const uint4 a = reinterpret_cast<const uint4*>(bs.gc)[2u * lane];
    const uint4 b = reinterpret_cast<const uint4*>(bs.gc)[2u * lane + 1u];
    const unsigned v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    const unsigned sum = a.x + a.y + a.z + a.w + b.x + b.y + b.z + b.w;
    unsigned before = wave_scan(sum) - sum;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      if (before < W && before + v[q] >= W) sh.digit = 8u * lane + unsigned(q);
      before += v[q];
    }
  }
  __syncthreads();
  const unsigned long long bw = (static_cast<unsigned long long>(sh.digit + 1u) << 32) | B;
  if (t == 0) __hip_atomic_store(word, bw, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return bw;
}

// LDS of the one-pass kernel.
struct OnePassShared {
  SelShared sh;
  unsigned start[kSelectMaxGatherSlots + 1];      // slot s holds positions [start[s], start[s+1])
  alignas(16) unsigned long long all[kRankCap + 128];  // survivors' composites, when they fit
                                                       // (+ a spare pair per lane)
  alignas(16) unsigned long long buck[kRankCap];  // the same, grouped by key bin
  alignas(16) unsigned long long top[kOnePassRankMax];  // the exact top W
  unsigned bstart[2048];                          // first position of each key bin in buck
  unsigned ntop;
  unsigned over[kThreads];                        // chunks with more than kSpecEntries survivors
  unsigned nover;
};

// Composite of a candidate: its key above its complemented flat index, so
// that one 64-bit comparison orders by score, then by lower index.
__device__ inline unsigned long long composite(uint2 e) {
  return (static_cast<unsigned long long>(e.x) << 32) | unsigned(~e.y);
}

// Writes out each of the m (<= kRankCap) composites in `c` (LDS) whose
// place among them -- the number of larger ones -- is below W.  The
// composites are grouped by a 2048-bin histogram of key - lo (bins in
// descending key order, so a bin's first position is the number of
// composites in the bins above it); a composite's place is then its bin's
// first position plus the larger composites of its own bin, which is
// usually a handful (all of them only when the keys are nearly equal).
template <bool BEAM>
__device__ inline void bucket_rank_emit(const SelectParams& p, OnePassShared& u, unsigned r,
                                        const unsigned long long* c, unsigned m,
                                        unsigned part = 0u, unsigned nparts = 1u) {
  SelShared& sh = u.sh;
  const unsigned t = threadIdx.x, lane = lane_id(), w = t >> 6;
  unsigned lo = ~0u, hi = 0u;
  for (unsigned q = t; q < m; q += kThreads) {
    const unsigned k = unsigned(c[q] >> 32);
    lo = min(lo, k);
    hi = max(hi, k);
  }
  const Red3 rr = block_reduce(sh, 0u, lo, hi);
  if (m == 0u) return;
  const int width = bit_width(rr.hi - rr.lo);
  const int shift = width > 11 ? width - 11 : 0;
  auto bin_of = [&](unsigned long long x) { return (unsigned(x >> 32) - rr.lo) >> shift; };
  reinterpret_cast<uint4*>(sh.hist)[t] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  for (unsigned q = t; q < m; q += kThreads) atomicAdd(&sh.hist[bin_of(c[q])], 1u);
  __syncthreads();
  {  // bstart[b] = composites in bins above b; thread t holds bins 2047 - 4t .. 2044 - 4t
    const uint4 h = reinterpret_cast<const uint4*>(sh.hist)[kThreads - 1 - t];
    const unsigned sum = h.x + h.y + h.z + h.w;
    const unsigned inc = wave_scan(sum);
    if (lane == 63) sh.red[0][w] = inc;
    __syncthreads();
    unsigned above = inc - sum;
#pragma unroll
    for (int w2 = 0; w2 < kWaves; ++w2) above += unsigned(w2) < w ? sh.red[0][w2] : 0u;
    const unsigned b0 = 2047u - 4u * t;
    u.bstart[b0] = above;
    u.bstart[b0 - 1u] = above + h.w;
    u.bstart[b0 - 2u] = above + h.w + h.z;
    u.bstart[b0 - 3u] = above + h.w + h.z + h.y;
  }
  __syncthreads();
  reinterpret_cast<uint4*>(sh.hist)[t] = make_uint4(0u, 0u, 0u, 0u);  // now per-bin cursors
  __syncthreads();
  for (unsigned q = t; q < m; q += kThreads) {
    const unsigned long long x = c[q];
    const unsigned b = bin_of(x);
    u.buck[u.bstart[b] + atomicAdd(&sh.hist[b], 1u)] = x;
  }
  __syncthreads();
  // this workgroup's share: composites part, part + nparts, ... of c (the
  // order within a bin of `buck` differs between workgroups, the order of c
  // does not), 16 lanes each (they split the bin's comparisons)
  const unsigned sub = t & 15u;
  for (unsigned k = t >> 4;; k += kThreads / 16u) {
    const unsigned q = part + nparts * k;
    if (part + nparts * (k - (t >> 4)) >= m) break;  // workgroup-uniform: no group has work
    const unsigned long long x = c[q < m ? q : 0u];
    const unsigned b = bin_of(x);
    const unsigned s0 = u.bstart[b], e0 = b > 0u ? u.bstart[b - 1u] : m;
    unsigned cnt = 0u;
    if (q < m)
      for (unsigned i = s0 + sub; i < e0; i += 16u) cnt += unsigned(u.buck[i] > x);
    cnt += dppu<0xB1>(cnt);   // quad_perm [1,0,3,2]
    cnt += dppu<0x4E>(cnt);   // quad_perm [2,3,0,1]
    cnt += dppu<0x141>(cnt);  // row_half_mirror
    cnt += dppu<0x140>(cnt);  // row_mirror
    if (sub == 0u && q < m && s0 + cnt < p.W) emit_pick<BEAM>(p, r, s0 + cnt, x);
  }
}

// The exact top W (W <= kOnePassRankMax <= n) of the n survivors of request
// r, read through get(q) in position (= index) order: radix passes of up to
// 11 bits over key - lo find the cut (every key above tau is in, and of the
// keys equal to tau the first `take` by position, or all keys >= tau when
// take = 0), the kept composites are collected in LDS, and each is placed by
// the number of larger ones.
template <bool BEAM, typename Get>
__device__ inline void onepass_topw(const SelectParams& p, OnePassShared& u, unsigned r,
                                    unsigned n, Get&& get) {
  const unsigned t = threadIdx.x, lane = lane_id(), w = t >> 6;
  SelShared& sh = u.sh;
  const unsigned W = p.W;
  unsigned tau = 0u, take = 0u;
  bool all_in = n <= W;
  if (!all_in) {
    unsigned lo = ~0u, hi = 0u;
    for (unsigned q = t; q < n; q += kThreads) {
      const unsigned k = unsigned(get(q) >> 32);
      lo = min(lo, k);
      hi = max(hi, k);
    }
    const Red3 rr = block_reduce(sh, 0u, lo, hi);
    if (rr.lo == rr.hi) {  // all equal: the first W by position
      tau = rr.lo;
      take = W;
    } else {
      int shift = bit_width(rr.hi - rr.lo);
      unsigned prefix = 0u, need = W;  // of key - lo
#pragma nounroll
      for (;;) {
        const int bits = shift < 11 ? shift : 11;
        shift -= bits;
        reinterpret_cast<uint4*>(sh.hist)[t] = make_uint4(0u, 0u, 0u, 0u);
        __syncthreads();
        const unsigned mask = (1u << bits) - 1u;
        for (unsigned q = t; q < n; q += kThreads) {
          const unsigned rel = unsigned(get(q) >> 32) - rr.lo;
          if (shr(rel, shift + bits) == prefix) atomicAdd(&sh.hist[(rel >> shift) & mask], 1u);
        }
        __syncthreads();
        find_bin(sh, need);
        prefix = (prefix << bits) | sh.digit;
        need = sh.need;
        const unsigned cnt = sh.cnt;
        if (cnt == need) {  // the boundary bin is taken whole
          tau = rr.lo + (prefix << shift);
          take = 0u;
          break;
        }
        if (shift == 0) {
          tau = rr.lo + prefix;
          take = need;
          break;
        }
      }
    }
  }
  if (t == 0) u.ntop = 0u;
  __syncthreads();
  unsigned eq_before = 0u;  // keys equal to tau at earlier positions
  for (unsigned base = 0u; base < n; base += kThreads) {
    const unsigned q = base + t;
    const bool valid = q < n;
    const unsigned long long c = valid ? get(q) : 0ull;
    const unsigned k = unsigned(c >> 32);
    bool sel = valid && (all_in || (take == 0u ? k >= tau : k > tau));
    if (take > 0u) {  // workgroup-uniform
      const bool eq = valid && k == tau;
      const unsigned long long be = __ballot(eq);
      if (lane == 0) sh.red[0][w] = unsigned(__popcll(be));
      __syncthreads();
      unsigned before = eq_before, round = 0u;
#pragma unroll
      for (int w2 = 0; w2 < kWaves; ++w2) {
        const unsigned x = sh.red[0][w2];
        round += x;
        before += unsigned(w2) < w ? x : 0u;
      }
      if (eq && before + mbcnt(be) < take) sel = true;
      eq_before += round;
      __syncthreads();  // sh.red is rewritten next round
    }
    if (sel) {
      const unsigned at = atomicAdd(&u.ntop, 1u);
      if (at < unsigned(kOnePassRankMax)) u.top[at] = c;
    }
  }
  __syncthreads();
  bucket_rank_emit<BEAM>(p, u, r, u.top, min(u.ntop, unsigned(kOnePassRankMax)));
}

// Final stage of request r in one of its nparts workgroups (every chunk's
// slot and (count, largest key) pair are stored).  One round of loads brings
// every chunk's count (thread t: chunk t, nchunks <= kThreads) and the first
// kSpecEntries entries of every slot (coalesced: a wave instruction covers 4
// slots, 16 lanes x 16 bytes each), which holds every survivor of most chunks;
// the survivors beyond them (a chunk holding many) are loaded by whole
// waves, one such chunk per wave at a time.  Up to kRankCap survivors are
// staged in LDS in position order; more are read from the slots on every
// pass of the exact top-W cut.
constexpr int kSpecEntries = 32;     // slot entries loaded with the counts
constexpr int kSpecRows = kThreads / 32;  // 32 slots per row of loads (8 waves x 4 slots)
constexpr int kBruteRankMax = 2048;  // survivors ranked by direct comparison
template <bool BEAM>
__device__ inline void onepass_final(const SelectParams& p, OnePassShared& u, unsigned r,
                                     unsigned part, unsigned nparts) {
  const unsigned ns = p.nwg, t = threadIdx.x;
  const unsigned lane = lane_id(), w = t >> 6;
  SelShared& sh = u.sh;
  const uint2* slots = p.cand_out + size_t(r) * ns * p.cap;
  const unsigned cnt = t < ns ? reinterpret_cast<const uint2*>(p.cnt_out)[size_t(r) * ns + t].x : 0u;
  uint4 ent[kSpecRows];  // entries 2 (lane % 16), + 1 of slot 32 i + 4 w + lane / 16
  // every row is issued (a load under a branch is waited for where the
  // branch joins, which would serialise the rows); rows beyond the request's
  // slots fall outside the buffer and read nothing
  {
    const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(slots, int(ns * p.cap * 8u));
#pragma unroll
    for (int i = 0; i < kSpecRows; ++i) {
      const unsigned c = unsigned(i) * 32u + 4u * w + (lane >> 4);
      ent[i] = __builtin_bit_cast(
          uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, (c * p.cap + 2u * (lane & 15u)) * 8u, 0, 0));
    }
  }
  if (t == 0) u.nover = 0u;
  const unsigned inc = wave_scan(cnt);
  if (lane == 63) sh.red[0][w] = inc;
  __syncthreads();
  unsigned start = inc - cnt, total = 0u;
#pragma unroll
  for (int w2 = 0; w2 < kWaves; ++w2) {
    const unsigned x = sh.red[0][w2];
    total += x;
    start += unsigned(w2) < w ? x : 0u;
  }
  // start[c] = total for every c >= ns (c <= kThreads), so that the slots
  // beyond the request's chunks read as empty
  u.start[t] = t < ns ? start : total;
  if (t == 0) u.start[kThreads] = total;
  if (cnt > unsigned(kSpecEntries)) u.over[atomicAdd(&u.nover, 1u)] = t;
  __syncthreads();
  if (total > unsigned(kRankCap)) {  // rare (heavy ties, or a bound that came late)
    // position q lies in the last slot whose start is <= q
    auto from_slots = [&](unsigned q) -> unsigned long long {
      unsigned lo = 0u, hi = ns;  // start[lo] <= q < start[hi]
      while (hi - lo > 1u) {
        const unsigned mid = (lo + hi) >> 1;
        if (u.start[mid] <= q) lo = mid;
        else hi = mid;
      }
      return composite(slots[size_t(lo) * p.cap + (q - u.start[lo])]);
    };
    if (part == 0u) onepass_topw<BEAM>(p, u, r, total, from_slots);
    return;
  }
  // starts of the rows' slots first (c < kThreads), then the writes of the
  // rows that hold chunks, unconditional: an entry past its slot's count
  // goes to a lane's own spare place after the staged range
  unsigned s0[kSpecRows], nn[kSpecRows];
#pragma unroll
  for (int i = 0; i < kSpecRows; ++i) {  // (no branch around reads: see the loads above)
    const unsigned c = unsigned(i) * 32u + 4u * w + (lane >> 4);
    s0[i] = u.start[c];
    nn[i] = u.start[c + 1] - s0[i];  // 0 beyond the request's chunks
  }
  const unsigned j = 2u * (lane & 15u), spare = unsigned(kRankCap) + 2u * lane;
#pragma unroll
  for (int i = 0; i < kSpecRows; ++i)
    if (unsigned(i) * 32u < ns) {
      u.all[j < nn[i] ? s0[i] + j : spare] = composite(make_uint2(ent[i].x, ent[i].y));
      u.all[j + 1u < nn[i] ? s0[i] + j + 1u : spare + 1u] = composite(make_uint2(ent[i].z, ent[i].w));
    }
  for (unsigned i = w; i < u.nover; i += kWaves) {  // wave-uniform
    const unsigned c = u.over[i], s0 = u.start[c], n = u.start[c + 1] - s0;
    const uint2* sl = slots + size_t(c) * p.cap;
    for (unsigned j0 = kSpecEntries; j0 < n; j0 += 512u) {  // 8 loads per lane in flight
      uint2 v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const unsigned jj = j0 + 64u * unsigned(k) + lane;
        v[k] = sl[jj < n ? jj : n - 1u];
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const unsigned jj = j0 + 64u * unsigned(k) + lane;
        if (jj < n) u.all[s0 + jj] = composite(v[k]);
      }
    }
  }
  __syncthreads();
  if (total > unsigned(kBruteRankMax)) {
    bucket_rank_emit<BEAM>(p, u, r, u.all, total, part, nparts);
    return;
  }
  // this workgroup's share: survivors part, part + nparts, ...; a survivor's
  // place is the number of larger composites.  A wave counts for two
  // survivors at once over interleaved pairs of positions, four pairs per
  // lane in flight (positions up to total + 511 < kRankCap are read; the ones
  // at or beyond total are not counted).
  for (unsigned k = 0;; k += 2u * kWaves) {
    if (part + nparts * k >= total) break;  // workgroup-uniform
    const unsigned q0 = part + nparts * (k + w), q1 = part + nparts * (k + kWaves + w);
    const unsigned long long x0 = u.all[q0 < total ? q0 : 0u], x1 = u.all[q1 < total ? q1 : 0u];
    unsigned c0 = 0u, c1 = 0u;
    for (unsigned j0 = 0; j0 < total; j0 += 512u) {
      ulonglong2 y[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        y[i] = *reinterpret_cast<const ulonglong2*>(&u.all[j0 + 128u * unsigned(i) + 2u * lane]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const unsigned j = j0 + 128u * unsigned(i) + 2u * lane;
        const bool v0 = j < total, v1 = j + 1u < total;
        c0 += unsigned(v0 && y[i].x > x0) + unsigned(v1 && y[i].y > x0);
        c1 += unsigned(v0 && y[i].x > x1) + unsigned(v1 && y[i].y > x1);
      }
    }
    const Red3 r0 = wave_reduce(c0, 0u, 0u), r1 = wave_reduce(c1, 0u, 0u);
    if (lane == 0u && q0 < total && r0.sum < p.W) emit_pick<BEAM>(p, r, r0.sum, x0);
    if (lane == 1u && q1 < total && r1.sum < p.W) emit_pick<BEAM>(p, r, r1.sum, x1);
  }
}

template <bool BEAM>
__global__ __launch_bounds__(kThreads) void select_onepass_kernel(SelectParams p) {
  __shared__ SelShared sh;
  __shared__ BoundShared bs;
  __shared__ unsigned long long bw_sh[1];
  __shared__ unsigned wmax[kWaves];
  const unsigned r = blockIdx.x / p.nwg, c = blockIdx.x - r * p.nwg;
  const unsigned base = c * unsigned(kSelectChunk);
  const unsigned n = min(p.N - base, unsigned(kSelectChunk));
  const unsigned t = threadIdx.x, w = t >> 6;
  const unsigned tag = p.ctl->epoch + 1u;  // (the final kernel advances the epoch)
  unsigned key[kNI];
  const unsigned vm = load_raw<BEAM>(p, r, base, n, key);
  if (t < (kNI * kWaves + 4) / 4) reinterpret_cast<uint4*>(sh.tab)[t] = make_uint4(0u, 0u, 0u, 0u);
  // 1. this wave's (M, m), published with the call's tag
  unsigned lmax = 0u;  // invalid slots hold key 0
#pragma unroll
  for (int i = 0; i < kNI; ++i) lmax = max(lmax, key[i]);
  const Red3 wr = wave_reduce(0u, (vm & 1u) ? lmax : ~0u, lmax);
  const unsigned km = unsigned(__popcll(__ballot((vm & 1u) && lmax == wr.hi)));
  if (lane_id() == 0) {
    st_agent4(p.ex, (r * p.nseg + c * kWaves + w) * 16u,
              make_uint4(wr.hi, wr.lo, km, tag ^ summary_mix(wr.hi, wr.lo, km)));
    wmax[w] = wr.hi;
  }
  // 2. the bound: computed by the request's first workgroup once every
  // summary is in, waited for by the others
  unsigned bound;  // keys below it are dropped
  unsigned long long* const word = &p.ctl->bound[r];
  if (c == 0u) {  // (chunk 0 is never above c*: its bound is B)
    uint4 e[kOnePassSegPer];
    const int late = onepass_poll(p, r, tag, e);
    bound = unsigned(onepass_bound(p, sh, bs, e, late, word));
  } else {
    if (t == 0) bw_sh[0] = wait_bound(word, p.wait_ticks, false);
    __syncthreads();
    unsigned long long bw = bw_sh[0];  // 0 after a timeout: no bound
    if (unsigned(bw >> 32) == kCstarPending) {
      // c* decides only for keys equal to B: a chunk holding none keeps the
      // keys >= B whichever side of c* it is on
      const unsigned B = unsigned(bw);
      int eq = 0;
#pragma unroll
      for (int i = 0; i < kNI; ++i) eq |= int(((vm >> i) & 1u) && key[i] == B);
      if (__syncthreads_or(eq)) {
        if (t == 0) bw_sh[0] = wait_bound(word, p.wait_ticks, true);
        __syncthreads();
        bw = bw_sh[0];
      }
    }
    const unsigned B = unsigned(bw), cstar = unsigned(bw >> 32) - 1u;
    bound = (c > cstar && B < ~0u) ? B + 1u : B;
  }
  // 3. survivors into the chunk's slot (as the filter kernel); the final
  // kernel reads them after this launch has ended
  unsigned keep = vm;
#pragma unroll
  for (int i = 0; i < kNI; ++i) keep &= ~(unsigned(key[i] < bound) << i);
  uint2* out = p.cand_out + (size_t(r) * p.nwg + c) * p.cap;
  auto put = [&](int i, unsigned rank) {
    out[rank] = make_uint2(key[i], base + unsigned(i) * kThreads + t);
  };
  unsigned total = ordered_plan_sparse(keep, sh);
  if (total > p.cap) {  // a chunk's exact top W of its survivors
    __syncthreads();
    keep = cut_mask(sh, key, keep, find_cut(sh, key, keep, p.W));
    total = replan_sparse(keep, sh);
    ordered_apply_sparse(keep, sh, put);
  } else {
    ordered_apply_sparse(keep, sh, put);
  }
  if (t == 0) {
    unsigned top = 0u;
#pragma unroll
    for (int w2 = 0; w2 < kWaves; ++w2) top = max(top, wmax[w2]);
    reinterpret_cast<uint2*>(p.cnt_out)[size_t(r) * p.nwg + c] = make_uint2(total, top);
  }
}

// Advances the epoch past this call's tag (workgroup 0 of the final kernel).
// After the largest tag it starts again at 0, and the summary region is
// cleared first, so that no summary left there carries a later call's tag.
__device__ inline void advance_epoch(const SelectParams& p) {
  const unsigned tag = p.ctl->epoch + 1u;
  __syncthreads();  // every thread has read it before thread 0 rewrites it
  if (tag == ~0u) {
    for (unsigned i = threadIdx.x; i < unsigned(kSelectSummaryBytes / 16); i += kThreads)
      p.ex[i] = make_uint4(0u, 0u, 0u, 0u);
  }
  if (threadIdx.x == 0) p.ctl->epoch = tag == ~0u ? 0u : tag;
}

// 4. fparts (<= kOnePassFinalParts) workgroups per request, after the pass: each stages
// all survivors and places its share of them; the first also returns the
// request's bound word to zero for the next call, and workgroup 0 advances
// the epoch.  (Without a control block, as after the two-pass filter, it
// only places.)
template <bool BEAM>
__global__ __launch_bounds__(kThreads) void select_onepass_final_kernel(SelectParams p) {
  __shared__ OnePassShared u;
  const unsigned r = blockIdx.x / p.fparts;
  const unsigned part = blockIdx.x - r * p.fparts;
  if (p.ctl != nullptr) {
    if (threadIdx.x == 0 && part == 0u) p.ctl->bound[r] = 0ull;
    if (blockIdx.x == 0u) advance_epoch(p);
  }
  onepass_final<BEAM>(p, u, r, part, p.fparts);
}


// Two-pass path, first pass with a bound (R <= kSelectOnePassMaxRequests and
// nseg <= kOnePassSegPer * kThreads): every wave publishes its one-pass
// summary (M, m, kM); the last workgroup of a request to finish (an arrival
// counter: no workgroup waits for another, so they need not all be resident
// at once) reads the request's summaries and writes its bound word, formed as
// in the one-pass path, for the filter pass.  The filter then compares with
// one word instead of forming a bound from every wave maximum in each of its
// workgroups.
template <bool BEAM, int ROWS>
__global__ __launch_bounds__(kThreads) void select_summary_kernel(SelectParams p) {
  __shared__ SelShared sh;
  __shared__ BoundShared bs;
  __shared__ unsigned last[1];
  const unsigned r = blockIdx.x / p.nwg, c = blockIdx.x - r * p.nwg;
  const unsigned base = c * unsigned(kSelectChunk);
  const unsigned n = min(p.N - base, unsigned(kSelectChunk));
  const unsigned t = threadIdx.x, w = t >> 6;
  unsigned key[kNI];
  const unsigned vm = load_raw<BEAM>(p, r, base, n, key);
  unsigned lmax = 0u;  // invalid slots hold key 0
#pragma unroll
  for (int i = 0; i < kNI; ++i) lmax = max(lmax, key[i]);
  const Red3 wr = wave_reduce(0u, (vm & 1u) ? lmax : ~0u, lmax);
  const unsigned km = unsigned(__popcll(__ballot((vm & 1u) && lmax == wr.hi)));
  if (lane_id() == 0)
    st_agent4(p.ex, (r * p.nseg + c * kWaves + w) * 16u, make_uint4(wr.hi, wr.lo, km, 0u));
  wait_stores();
  __syncthreads();
  if (t == 0) last[0] = atomicAdd(&p.ctl->arrive[r], 1u) == p.nwg - 1u;
  __syncthreads();
  if (last[0] == 0u) return;  // workgroup-uniform
  uint4 e[ROWS];  // (nseg <= ROWS * kThreads)
  const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(p.ex + size_t(r) * p.nseg, int(p.nseg * 16u));
#pragma unroll
  for (int i = 0; i < ROWS; ++i) e[i] = ld_agent4(rs, (unsigned(i) * kThreads + t) * 16u);
  onepass_bound<ROWS>(p, sh, bs, e, 0, &p.tp_bound[r]);
  if (t == 0) p.ctl->arrive[r] = 0u;
}

// Workgroups of the one-pass kernel that can be resident at once on the
// current device (all of a call's workgroups must be, or they would wait on
// ones that cannot start), and its wait for the bound in wall-clock ticks;
// both queried once per device.
struct OnePassDevice {
  unsigned capacity;
  unsigned long long wait_ticks;
};
OnePassDevice onepass_device() {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static OnePassDevice cache[kMaxDevices] = {};
  static bool known[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return {0u, 0ull};
  std::lock_guard<std::mutex> lock(mu);
  if (!known[dev]) {
    OnePassDevice d{0u, 0ull};
    int cus = 0, per_cu_a = 0, per_cu_b = 0, khz = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &per_cu_a, reinterpret_cast<const void*>(select_onepass_kernel<true>), kThreads, 0) ==
            hipSuccess &&
        hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &per_cu_b, reinterpret_cast<const void*>(select_onepass_kernel<false>), kThreads, 0) ==
            hipSuccess &&
        hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) == hipSuccess &&
        cus > 0 && khz > 0) {
      d.capacity = unsigned(cus) * unsigned(std::min(per_cu_a, per_cu_b));
      d.wait_ticks = 20ull * unsigned(khz) / 1000ull;  // 20 us
    }
    cache[dev] = d;
    known[dev] = true;
  }
  return cache[dev];
}
unsigned onepass_capacity() { return onepass_device().capacity; }
unsigned long long onepass_wait_ticks() { return onepass_device().wait_ticks; }

}  // namespace

hipError_t launch_select(const SelectPlan& plan, int R, int prev_width, int vocab, int width,
                         const float* logp, const float* beam, int* parents, int* tokens,
                         float* scores, void* workspace, hipStream_t st) {
  SelectParams p{};
  p.logp = logp;
  p.beam = beam;
  p.parents = parents;
  p.tokens = tokens;
  p.scores = scores;
  p.V = unsigned(vocab);
  p.W_prev = unsigned(prev_width);
  p.N = p.V * p.W_prev;
  p.W = unsigned(width);
  p.cap = plan.cap;
  p.lcap = unsigned(__builtin_ctz(plan.cap));
  p.group = plan.group;
  p.inv_v = 1.0 / double(vocab);
  char* ws = static_cast<char*>(workspace);
  const bool has_beam = beam != nullptr;
  if (plan.two_pass && R <= kSelectOnePassMaxRequests && width <= kOnePassRankMax &&
      plan.nseg <= unsigned(kOnePassSegPer * kThreads) &&
      size_t(R) * plan.nseg * 16u <= kSelectSummaryBytes &&
      unsigned(R) * plan.nchunks <= onepass_capacity()) {
    p.ctl = reinterpret_cast<OnePassCtl*>(ws);
    p.ex = reinterpret_cast<uint4*>(ws + kSelectCtlBytes);
    p.nseg = plan.nseg;
    p.nwg = plan.nchunks;
    p.cand_out = reinterpret_cast<uint2*>(ws + plan.slot_off);
    p.cnt_out = reinterpret_cast<unsigned*>(ws + plan.cnt_off);
    p.wait_ticks = onepass_wait_ticks();
    const unsigned blocks = unsigned(R) * plan.nchunks;
    if (has_beam) select_onepass_kernel<true><<<blocks, kThreads, 0, st>>>(p);
    else select_onepass_kernel<false><<<blocks, kThreads, 0, st>>>(p);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // a share of survivors per workgroup, the whole call in about one round of
    // workgroups (one per compute unit)
    p.fparts = std::max(1u, std::min(unsigned(kOnePassFinalParts), 256u / unsigned(R)));
    const unsigned fblocks = unsigned(R) * p.fparts;
    if (has_beam) select_onepass_final_kernel<true><<<fblocks, kThreads, 0, st>>>(p);
    else select_onepass_final_kernel<false><<<fblocks, kThreads, 0, st>>>(p);
    return hipGetLastError();
  }
  if (plan.two_pass) {
    p.nseg = plan.nseg;
    p.nwg = plan.nchunks;
    p.cand_out = reinterpret_cast<uint2*>(ws + plan.slot_off);
    p.cnt_out = reinterpret_cast<unsigned*>(ws + plan.cnt_off);
    const unsigned blocks = unsigned(R) * plan.nchunks;
    if (R <= kSelectOnePassMaxRequests && plan.nseg <= unsigned(kOnePassSegPer * kThreads) &&
        unsigned(R) * plan.nchunks >= 4u * onepass_capacity()) {
      // summaries and one bound word per request (the arrival counters are
      // in the control block).  The summary pass costs about 10 us more than
      // the wave maxima (each workgroup waits for its stores and its arrival
      // before it leaves; the last request's bound ends the launch), and it
      // saves the filter's per-workgroup bound (about 3.5 us per round of
      // workgroups on the chip): it pays from four rounds on.
      p.ctl = reinterpret_cast<OnePassCtl*>(ws);
      p.ex = reinterpret_cast<uint4*>(ws + plan.seg_off);
      p.tp_bound = reinterpret_cast<unsigned long long*>(ws + plan.bound_off);
      // (the bound's rows of summaries per thread: as few as hold nseg)
      if (plan.nseg <= 2u * kThreads) {
        if (has_beam) select_summary_kernel<true, 2><<<blocks, kThreads, 0, st>>>(p);
        else select_summary_kernel<false, 2><<<blocks, kThreads, 0, st>>>(p);
      } else if (plan.nseg <= 4u * kThreads) {
        if (has_beam) select_summary_kernel<true, 4><<<blocks, kThreads, 0, st>>>(p);
        else select_summary_kernel<false, 4><<<blocks, kThreads, 0, st>>>(p);
      } else {
        if (has_beam) select_summary_kernel<true, kOnePassSegPer><<<blocks, kThreads, 0, st>>>(p);
        else select_summary_kernel<false, kOnePassSegPer><<<blocks, kThreads, 0, st>>>(p);
      }
    } else {
      p.segmax = reinterpret_cast<unsigned*>(ws + plan.seg_off);
      if (has_beam) select_segmax_kernel<true><<<blocks, kThreads, 0, st>>>(p);
      else select_segmax_kernel<false><<<blocks, kThreads, 0, st>>>(p);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (p.tp_bound != nullptr) {
      if (has_beam) select_filter_kernel<true, true><<<blocks, kThreads, 0, st>>>(p);
      else select_filter_kernel<false, true><<<blocks, kThreads, 0, st>>>(p);
    } else {
      if (has_beam) select_filter_kernel<true, false><<<blocks, kThreads, 0, st>>>(p);
      else select_filter_kernel<false, false><<<blocks, kThreads, 0, st>>>(p);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (plan.nchunks <= unsigned(kThreads) && p.W <= unsigned(kOnePassRankMax)) {
      // the filter's slots have the one-pass layout: the one-pass placing
      // kernel ranks them (no control block: R may exceed its requests)
      p.ctl = nullptr;
      p.fparts = std::max(1u, std::min(unsigned(kOnePassFinalParts), 256u / unsigned(R)));
      const unsigned fblocks = unsigned(R) * p.fparts;
      if (has_beam) select_onepass_final_kernel<true><<<fblocks, kThreads, 0, st>>>(p);
      else select_onepass_final_kernel<false><<<fblocks, kThreads, 0, st>>>(p);
      return hipGetLastError();
    }
    p.cand_in = p.cand_out;
    p.cnt_in = p.cnt_out;
    p.nslots_in = plan.nchunks;
    const unsigned rblocks = unsigned(R) * kRankBlocks;
    if (has_beam) select_rank_kernel<true><<<rblocks, kThreads, 0, st>>>(p);
    else select_rank_kernel<false><<<rblocks, kThreads, 0, st>>>(p);
    return hipGetLastError();
  }
  for (int s = 0; s < plan.stages; ++s) {
    const int in = (s - 1) & 1, out = s & 1;
    p.cand_in = s == 0 ? nullptr : reinterpret_cast<const uint2*>(ws + plan.pair_off[in]);
    p.cnt_in = s == 0 ? nullptr : reinterpret_cast<const unsigned*>(ws + plan.count_off[in]);
    p.cand_out = reinterpret_cast<uint2*>(ws + plan.pair_off[out]);
    p.cnt_out = reinterpret_cast<unsigned*>(ws + plan.count_off[out]);
    p.nslots_in = s == 0 ? 0u : plan.nin[s];
    p.nwg = plan.nwg[s];
    const unsigned blocks = unsigned(R) * plan.nwg[s];
    if (s == 0) {
      if (has_beam) select_raw_stage_kernel<true><<<blocks, kThreads, 0, st>>>(p);
      else select_raw_stage_kernel<false><<<blocks, kThreads, 0, st>>>(p);
    } else {
      select_slot_stage_kernel<<<blocks, kThreads, 0, st>>>(p);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int last = (plan.stages - 1) & 1;
  p.cand_in =
      plan.stages == 0 ? nullptr : reinterpret_cast<const uint2*>(ws + plan.pair_off[last]);
  p.cnt_in =
      plan.stages == 0 ? nullptr : reinterpret_cast<const unsigned*>(ws + plan.count_off[last]);
  p.cand_out = nullptr;
  p.cnt_out = nullptr;
  p.nslots_in = plan.stages == 0 ? 0u : plan.final_in;
  p.nwg = 1;
  if (plan.stages == 0) {
    if (has_beam) select_final_kernel<true, true><<<R, kThreads, 0, st>>>(p);
    else select_final_kernel<true, false><<<R, kThreads, 0, st>>>(p);
  } else {
    if (has_beam) select_final_kernel<false, true><<<R, kThreads, 0, st>>>(p);
    else select_final_kernel<false, false><<<R, kThreads, 0, st>>>(p);
  }
  return hipGetLastError();
}

// Device address of this GPU's scratch array (looked up once per device, with
// that device current; each GPU holds its own copy at its own address).
hipError_t select_scratch(void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* cache[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!cache[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    cache[dev] = p;
  }
  *out = cache[dev];
  return hipSuccess;
}

}  // namespace onela
