// Global top-W beam selection (Sec. 2.1) on gfx950.
//
// Every live beam p of a request is expanded over the V codebook entries; the
// candidate (p, v) has score  beam[p] + logp[p][v]  (one fp32 rounding; logp
// alone when no beam scores are given) and flat index p * V + v.  The W best
// candidates are kept, best first.  The order is total: higher score first,
// equal scores by lower flat index, -0.0 below +0.0, every NaN below every
// number.  It is realised on an unsigned 32-bit key that is monotone in the
// score (sign-magnitude flip; all NaNs map to 0) plus the flat index.
//
// The work is HBM-bound (N = W_prev * V fp32 scores per request, read once),
// so it is organised as a reduction tree of exact selections rather than a
// global sort:
//   * stage kernel: one 512-thread workgroup per chunk of 16384 candidates
//     keeps that chunk's top min(W, n) candidates, written as (key, index)
//     pairs in index order.  Any candidate of the global top W is in the
//     top W of its own chunk, so each stage shrinks the set by 16384 / W
//     without losing one.
//   * final kernel: one workgroup per request selects the top W of the last
//     <= 16384 candidates, sorts them (bitonic, in LDS) and writes parents,
//     tokens and scores.
// Inside a workgroup, selection is a three-pass radix select on the key
// (11 + 11 + 10 bits) with LDS histograms; the boundary key's ties are
// resolved by an index-ordered scan (ballot + mbcnt per wave, one 256-entry
// scan across (element slot, wave)), so the result is deterministic and needs
// no global atomics.
#include "internal.h"

namespace onela {
namespace {

constexpr int kThreads = kSelectThreads;
constexpr int kWaves = kThreads / 64;
constexpr int kNI = kSelectChunk / kThreads;  // candidates per thread
static_assert(kNI * kWaves == 256, "the index-ordered scan covers 256 (slot, wave) entries");

struct SelectParams {
  const float* logp;     // [R][N] log-probabilities, N = W_prev * V
  const float* beam;     // [R][W_prev] beam scores, or null
  const uint2* cand_in;  // [R][n_in] (key, flat index) pairs in index order; null: read logp
  uint2* cand_out;       // [R][out_stride] (stage kernel)
  int* parents;          // [R][W] (final kernel)
  int* tokens;
  float* scores;
  unsigned N, V, W_prev;
  unsigned n_in;        // input candidates per request
  unsigned nchunks;     // chunks per request (stage kernel)
  unsigned out_stride;  // output pairs per request (stage kernel)
  unsigned W;
  double inv_v;  // 1 / V
};

struct alignas(16) SelShared {
  unsigned hist[2048];
  unsigned tab[kNI * kWaves + 4];
  unsigned wsum[kWaves];
  unsigned digit, need, cnt;
};

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

template <bool BEAM>
__device__ inline float candidate_score(const float* logp_r, const float* beam_r, unsigned idx,
                                        unsigned V, double inv_v) {
  const float x = logp_r[idx];
  if constexpr (BEAM) return beam_r[row_of(idx, V, inv_v)] + x;
  return x;
}

__device__ inline unsigned lane_id() { return threadIdx.x & 63; }

__device__ inline unsigned mbcnt(unsigned long long m) {
  return __builtin_amdgcn_mbcnt_hi(unsigned(m >> 32), __builtin_amdgcn_mbcnt_lo(unsigned(m), 0u));
}

// hist[bin] += 1 for every lane with act.  The two most frequent cases of
// many lanes hitting one bin (narrow score distributions) are aggregated with
// a ballot so that one lane adds the count; the rest use LDS atomics.  Must be
// reached by all lanes of the wave.
__device__ inline void hist_add(unsigned* hist, unsigned bin, bool act) {
  unsigned long long pend = __ballot(act);
#pragma unroll
  for (int round = 0; round < 2; ++round) {
    if (pend == 0) return;
    const int leader = __builtin_ctzll(pend);
    const unsigned b = __builtin_amdgcn_readlane(bin, leader);
    const unsigned long long same = __ballot(act && bin == b);
    if (lane_id() == unsigned(leader)) atomicAdd(&hist[b], unsigned(__popcll(same)));
    if (bin == b) act = false;
    pend &= ~same;
  }
  if (act) atomicAdd(&hist[bin], 1u);
}

// After a histogram pass: the bin where the running count from the top first
// reaches `need`.  Publishes (digit, need - count above it, bin count).
__device__ inline void find_bin(SelShared& sh, unsigned need) {
  const unsigned t = threadIdx.x, lane = lane_id(), w = t >> 6;
  const uint4 h = reinterpret_cast<const uint4*>(sh.hist)[t];  // bins 4t .. 4t+3
  const unsigned s = h.x + h.y + h.z + h.w;
  unsigned suf = s;  // sum over lanes >= lane of this wave
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const unsigned y = __shfl_down(suf, d);
    if (lane + d < 64) suf += y;
  }
  if (lane == 0) sh.wsum[w] = suf;
  __syncthreads();
  unsigned above = suf - s;
  for (unsigned w2 = w + 1; w2 < unsigned(kWaves); ++w2) above += sh.wsum[w2];
  const unsigned hb[4] = {h.x, h.y, h.z, h.w};
#pragma unroll
  for (int b = 3; b >= 0; --b) {
    if (above < need && need <= above + hb[b]) {
      sh.digit = 4 * t + b;
      sh.need = need - above;
      sh.cnt = hb[b];
    }
    above += hb[b];
  }
  __syncthreads();
}

// Calls fn(i, offset) for every flagged element (bit i of f: element i),
// where offset is its exclusive rank among the flagged elements of the
// workgroup in index order; element i of a thread sits at chunk position
// i * kThreads + threadIdx.x.  Wave-local ranks come from ballot + mbcnt and
// are kept packed 4 per register; one wave scans the 256 (slot, wave) counts.
template <typename F>
__device__ inline void for_each_ordered(unsigned f, SelShared& sh, F&& fn) {
  const unsigned lane = lane_id(), w = threadIdx.x >> 6;
  unsigned pre[kNI / 4];
#pragma unroll
  for (int i = 0; i < kNI; ++i) {
    const unsigned long long b = __ballot((f >> i) & 1u);
    const unsigned m = mbcnt(b);
    pre[i / 4] = (i % 4 == 0) ? m : (pre[i / 4] | (m << (8 * (i % 4))));
    if (lane == 0) sh.tab[i * kWaves + w] = unsigned(__popcll(b));
  }
  __syncthreads();
  if (w == 0) {
    const uint4 v = reinterpret_cast<const uint4*>(sh.tab)[lane];
    const unsigned s = v.x + v.y + v.z + v.w;
    unsigned inc = s;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const unsigned y = __shfl_up(inc, d);
      if (lane >= unsigned(d)) inc += y;
    }
    const unsigned ex = inc - s;
    reinterpret_cast<uint4*>(sh.tab)[lane] =
        make_uint4(ex, ex + v.x, ex + v.x + v.y, ex + v.x + v.y + v.z);
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kNI; ++i)
    if ((f >> i) & 1u) fn(i, sh.tab[i * kWaves + w] + ((pre[i / 4] >> (8 * (i % 4))) & 0xffu));
  __syncthreads();
}

// One radix pass over the keys whose bits above `shift + bits` equal the
// prefix found so far.
template <int SHIFT, int BITS, int PSHIFT>
__device__ inline void radix_pass(SelShared& sh, const unsigned (&key)[kNI], int nv,
                                  unsigned prefix, unsigned need) {
  reinterpret_cast<uint4*>(sh.hist)[threadIdx.x] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kNI; ++i) {
    bool act = i < nv;
    if constexpr (PSHIFT < 32) act = act && (key[i] >> PSHIFT) == prefix;
    hist_add(sh.hist, (key[i] >> SHIFT) & ((1u << BITS) - 1u), act);
  }
  __syncthreads();
  find_bin(sh, need);
}

// Flags (bit i: element i) the top `need0` elements of the workgroup's chunk
// (key order, ties by chunk position).
__device__ inline unsigned select_top(SelShared& sh, const unsigned (&key)[kNI], int nv,
                                      unsigned need0) {
  radix_pass<21, 11, 32>(sh, key, nv, 0u, need0);
  unsigned prefix = sh.digit, need = sh.need;
  radix_pass<10, 11, 21>(sh, key, nv, prefix, need);
  prefix = (prefix << 11) | sh.digit;
  need = sh.need;
  radix_pass<0, 10, 10>(sh, key, nv, prefix, need);
  const unsigned tau = (prefix << 10) | sh.digit;
  need = sh.need;
  const unsigned ties = sh.cnt;
  unsigned gt = 0u, eq = 0u;
#pragma unroll
  for (int i = 0; i < kNI; ++i) {
    gt |= unsigned(i < nv && key[i] > tau) << i;
    eq |= unsigned(i < nv && key[i] == tau) << i;
  }
  if (ties > need) {  // keep the first `need` ties in index order
    unsigned drop = 0u;
    for_each_ordered(eq, sh, [&](int i, unsigned o) { drop |= unsigned(o >= need) << i; });
    eq &= ~drop;
  }
  return gt | eq;
}

// Keys of the candidates at chunk positions [base, base + n) of request r;
// for pair input also their flat indices (raw input: index = position).
template <bool RAW, bool BEAM>
__device__ inline void load_chunk(const SelectParams& p, unsigned r, unsigned base, int nv,
                                  unsigned (&key)[kNI], unsigned (&idx)[kNI]) {
  const float* logp_r = p.logp + size_t(r) * p.N;
  const float* beam_r = BEAM ? p.beam + size_t(r) * p.W_prev : nullptr;
  const uint2* cand_r = RAW ? nullptr : p.cand_in + size_t(r) * p.n_in;
#pragma unroll
  for (int i = 0; i < kNI; ++i) {
    const unsigned pos = base + unsigned(i) * kThreads + threadIdx.x;
    key[i] = 0u;
    if constexpr (!RAW) idx[i] = 0u;
    if (i < nv) {
      if constexpr (RAW) {
        key[i] = order_key(candidate_score<BEAM>(logp_r, beam_r, pos, p.V, p.inv_v));
      } else {
        const uint2 c = cand_r[pos];
        key[i] = c.x;
        idx[i] = c.y;
      }
    }
  }
}

__device__ inline int valid_per_thread(unsigned n) {
  const unsigned t = threadIdx.x;
  return n > t ? int((n - t + kThreads - 1) / kThreads) : 0;
}

template <bool RAW, bool BEAM>
__global__ __launch_bounds__(kThreads) void select_stage_kernel(SelectParams p) {
  __shared__ SelShared sh;
  const unsigned r = blockIdx.x / p.nchunks, c = blockIdx.x - r * p.nchunks;
  const unsigned base = c * unsigned(kSelectChunk);
  const unsigned n = min(p.n_in - base, unsigned(kSelectChunk));
  const int nv = valid_per_thread(n);
  unsigned key[kNI], idx[kNI];
  load_chunk<RAW, BEAM>(p, r, base, nv, key, idx);
  const unsigned sel = select_top(sh, key, nv, min(p.W, n));
  uint2* out = p.cand_out + size_t(r) * p.out_stride + size_t(c) * p.W;
  for_each_ordered(sel, sh, [&](int i, unsigned o) {
    const unsigned fi = RAW ? base + unsigned(i) * kThreads + threadIdx.x : idx[i];
    out[o] = make_uint2(key[i], fi);
  });
}

template <bool RAW, bool BEAM>
__global__ __launch_bounds__(kThreads) void select_final_kernel(SelectParams p) {
  __shared__ SelShared sh;
  __shared__ unsigned long long srt[kSelectMaxWidth];
  const unsigned r = blockIdx.x;
  const int nv = valid_per_thread(p.n_in);
  unsigned key[kNI], idx[kNI];
  load_chunk<RAW, BEAM>(p, r, 0u, nv, key, idx);
  const unsigned sel = select_top(sh, key, nv, p.W);
  // Composite sort key: score key high, complemented index low, so that the
  // descending order is (score desc, index asc).  Padding (0) sorts last.
  for_each_ordered(sel, sh, [&](int i, unsigned o) {
    const unsigned fi = RAW ? unsigned(i) * kThreads + threadIdx.x : idx[i];
    srt[o] = (static_cast<unsigned long long>(key[i]) << 32) | unsigned(~fi);
  });
  unsigned n2 = 1;
  while (n2 < p.W) n2 <<= 1;
  for (unsigned j = p.W + threadIdx.x; j < n2; j += kThreads) srt[j] = 0ull;
  __syncthreads();
  for (unsigned k = 2; k <= n2; k <<= 1) {
    for (unsigned j = k >> 1; j > 0; j >>= 1) {
      for (unsigned x = threadIdx.x; x < n2 / 2; x += kThreads) {
        const unsigned a = 2 * x - (x & (j - 1)), b = a + j;
        const unsigned long long va = srt[a], vb = srt[b];
        const bool desc = (a & k) == 0;
        if (desc ? va < vb : va > vb) {
          srt[a] = vb;
          srt[b] = va;
        }
      }
      __syncthreads();
    }
  }
  const float* logp_r = p.logp + size_t(r) * p.N;
  for (unsigned j = threadIdx.x; j < p.W; j += kThreads) {
    const unsigned fi = ~unsigned(srt[j]);
    const unsigned row = row_of(fi, p.V, p.inv_v);
    const size_t o = size_t(r) * p.W + j;
    p.parents[o] = int(row);
    p.tokens[o] = int(fi - row * p.V);
    if constexpr (BEAM) p.scores[o] = p.beam[size_t(r) * p.W_prev + row] + logp_r[fi];
    else p.scores[o] = logp_r[fi];
  }
}

template <bool RAW>
void launch_stage(const SelectParams& p, unsigned blocks, bool beam, hipStream_t st) {
  if (beam) select_stage_kernel<RAW, true><<<blocks, kThreads, 0, st>>>(p);
  else select_stage_kernel<RAW, false><<<blocks, kThreads, 0, st>>>(p);
}

template <bool RAW>
void launch_final(const SelectParams& p, unsigned blocks, bool beam, hipStream_t st) {
  if (beam) select_final_kernel<RAW, true><<<blocks, kThreads, 0, st>>>(p);
  else select_final_kernel<RAW, false><<<blocks, kThreads, 0, st>>>(p);
}

}  // namespace

bool select_plan(int R, unsigned N, unsigned W, SelectPlan* plan) {
  *plan = SelectPlan{};
  if (R < 1 || N < 1 || W < 1 || W > N || W > unsigned(kSelectMaxWidth) ||
      N > kSelectMaxCandidates)
    return false;
  size_t buf[2] = {0, 0};
  unsigned n = N;
  int s = 0;
  while (n > unsigned(kSelectChunk)) {
    if (s == kSelectMaxStages) return false;
    const unsigned chunks = (n + kSelectChunk - 1) / kSelectChunk;
    const unsigned last = n - (chunks - 1) * unsigned(kSelectChunk);
    const unsigned out = (chunks - 1) * W + (last < W ? last : W);
    plan->n[s] = n;
    plan->chunks[s] = chunks;
    plan->out[s] = out;
    const size_t bytes = size_t(R) * out * sizeof(uint2);
    if (bytes > buf[s & 1]) buf[s & 1] = bytes;
    n = out;
    ++s;
  }
  plan->stages = s;
  plan->n_final = n;
  auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
  plan->buf_bytes[0] = up(buf[0]);
  plan->buf_bytes[1] = up(buf[1]);
  plan->total = plan->buf_bytes[0] + plan->buf_bytes[1];
  return true;
}

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
  p.inv_v = 1.0 / double(vocab);
  uint2* bufs[2] = {static_cast<uint2*>(workspace),
                    reinterpret_cast<uint2*>(static_cast<char*>(workspace) + plan.buf_bytes[0])};
  const bool has_beam = beam != nullptr;
  for (int s = 0; s < plan.stages; ++s) {
    p.cand_in = s == 0 ? nullptr : bufs[(s - 1) & 1];
    p.cand_out = bufs[s & 1];
    p.n_in = plan.n[s];
    p.nchunks = plan.chunks[s];
    p.out_stride = plan.out[s];
    const unsigned blocks = unsigned(R) * plan.chunks[s];
    if (s == 0) launch_stage<true>(p, blocks, has_beam, st);
    else launch_stage<false>(p, blocks, false, st);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  p.cand_in = plan.stages == 0 ? nullptr : bufs[(plan.stages - 1) & 1];
  p.cand_out = nullptr;
  p.n_in = plan.n_final;
  p.nchunks = 1;
  p.out_stride = 0;
  if (plan.stages == 0) launch_final<true>(p, unsigned(R), has_beam, st);
  else launch_final<false>(p, unsigned(R), has_beam, st);
  return hipGetLastError();
}

}  // namespace onela
