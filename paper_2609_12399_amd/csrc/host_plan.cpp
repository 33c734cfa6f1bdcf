// Host-side plans and checks of libonela (see host_plan.h): plain C++, no
// HIP, built into the library and, on its own, under the host sanitizers.
#include "host_plan.h"

#include <algorithm>

namespace onela {

namespace {
size_t round256(size_t x) { return (x + 255) & ~size_t(255); }

unsigned pow2_ceil(unsigned x) {
  unsigned y = 1;
  while (y < x) y <<= 1;
  return y;
}
}  // namespace

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

bool decode_supported(const Shape& s) {
  const int dk = s.dk, dv = s.dv;
  if ((dk == 32 && dv == 32) || (dk == 64 && dv == 64) || (dk == 128 && dv == 128)) return true;
  if (!s.bf16) return false;
  return (dk == 128 && (dv == 256 || dv == 512)) || (dk == 256 && (dv == 256 || dv == 512));
}

onela_status_t shape_of(const onela_config_t* c, Shape* s) {
  if (!c) return ONELA_EINVAL;
  if (c->num_requests < 1 || c->num_qk_heads < 1 || c->num_v_heads < 1)
    return ONELA_EINVAL;
  if (c->num_v_heads % c->num_qk_heads) return ONELA_EINVAL;
  if (c->max_beams < 1 || c->max_beams > 65536) return ONELA_EINVAL;
  if (c->max_steps < 1 || c->max_steps > kMaxSteps) return ONELA_EINVAL;
  if (c->io_dtype != ONELA_F32 && c->io_dtype != ONELA_BF16) return ONELA_EINVAL;
  if (c->record_kind != ONELA_RECORD_INPUTS && c->record_kind != ONELA_RECORD_DELTA)
    return ONELA_EINVAL;
  if (c->record_storage != ONELA_RECORDS_COPY && c->record_storage != ONELA_RECORDS_BORROW)
    return ONELA_EINVAL;
  if (c->record_storage == ONELA_RECORDS_BORROW && c->record_kind == ONELA_RECORD_DELTA)
    return ONELA_EINVAL;
  Shape t{c->num_requests, c->num_qk_heads, c->num_v_heads,
          c->d_k,          c->d_v,          c->max_beams,
          c->max_steps,    c->io_dtype == ONELA_BF16, c->record_kind == ONELA_RECORD_DELTA,
          c->record_storage == ONELA_RECORDS_BORROW};
  if (!decode_supported(t)) return ONELA_EINVAL;
  // the kernels form 32-bit byte offsets: every region must stay below 2 GiB
  const double big = double(t.R) * t.tmax * (t.HV > t.HK ? t.HV : t.HK) * t.wmax *
                     (t.dv > t.dk ? t.dv : t.dk) * t.io_bytes();
  const double outb = double(t.R) * t.wmax * t.HV * t.dv * 4.0;
  const double s0b = double(t.R) * t.HV * t.dv * t.dk * 4.0;
  if (big >= 2147483648.0 || outb >= 2147483648.0 || s0b >= 2147483648.0) return ONELA_EINVAL;
  *s = t;
  return ONELA_OK;
}


Layout layout_of(const Shape& s) {
  Layout l{};
  const size_t R = s.R, T = s.tmax, W = s.wmax;
  l.status = 256;
  l.anc = round256(sizeof(int) * R * W * T);
  l.s_frag = round256(sizeof(uint16_t) * 2 * R * s.HV * size_t(s.dv) * s.dk);
  const size_t arena = s.borrow ? 0 : 1;  // borrowed records need no arena
  l.k = arena * round256(size_t(s.io_bytes()) * R * T * s.HK * W * s.dk);
  l.v = arena * round256(size_t(s.io_bytes()) * R * T * s.HV * W * s.dv);
  l.ab = arena * round256(2 * sizeof(float) * R * T * s.HV * W);
  l.d = s.delta ? l.v : 0;  // delta rows take the size of input v rows (fp16 / fp32)
  l.ds = s.delta ? round256(sizeof(unsigned) * R * T * s.HV * W) : 0;  // delta row scales
  l.total = l.status + 2 * l.anc + l.s_frag + l.k + l.v + l.ab + l.d + l.ds;
  return l;
}


size_t prefill_chunked_workspace_bytes(const Shape& s, int prompt_len) {
  const size_t nch = size_t(prompt_len + kPrefillChunk - 1) / kPrefillChunk;
  const size_t per = size_t(kPrefillChunk) * (2 * s.dk + s.dv) * sizeof(float);
  auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
  const size_t units = size_t(s.R) * s.HV;
  return up(units * nch * per) + up(units * nch * 16 * sizeof(float));
}

bool select_plan(int R, unsigned N, unsigned W, SelectPlan* plan) {
  *plan = SelectPlan{};
  if (R < 1 || N < 1 || W < 1 || W > N || W > unsigned(kSelectMaxWidth) ||
      N > kSelectMaxCandidates)
    return false;
  // Slot capacity: room for about twice the kept count, at least 64, at most
  // a quarter of a workgroup's candidates (never below W).
  unsigned cap = pow2_ceil(2 * W);
  if (cap < 64) cap = 64;
  if (cap > unsigned(kSelectChunk) / 4) cap = std::max(unsigned(kSelectChunk) / 4, pow2_ceil(W));
  plan->cap = cap;
  plan->group = unsigned(kSelectChunk) / cap;
  auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
  const unsigned nchunks = (N + kSelectChunk - 1) / kSelectChunk;
  // Every plan starts with the one-pass path's control block and summary
  // region, which no other data overwrites, so that a workspace shared by
  // calls of any shape keeps the state the one-pass path carries from call
  // to call.
  const size_t ctl = kSelectCtlBytes + kSelectSummaryBytes;
  // Two-pass path: enough wave maxima (2048 candidates each) for a tight
  // bound, few enough chunks for the one-workgroup gather.
  if (N > unsigned(kSelectChunk) && uint64_t(N) >= uint64_t(2) * W * 2048u &&
      nchunks <= unsigned(kSelectMaxGatherSlots)) {
    plan->two_pass = true;
    plan->nchunks = nchunks;
    plan->nseg = nchunks * (kSelectThreads / 64);
    plan->seg_off = ctl;  // [R][nseg] wave summaries (M, m, kM, 0), or uint32 maxima
    plan->bound_off = ctl + up(size_t(R) * plan->nseg * 16);  // [R] bound words
    plan->slot_off = plan->bound_off + up(size_t(R) * 8);
    plan->cnt_off = plan->slot_off + up(size_t(R) * nchunks * cap * 8 /* (key, index) */);
    plan->total = plan->cnt_off + up(size_t(R) * nchunks * 8 /* (count, largest key) */);
    return true;
  }
  size_t pairs[2] = {0, 0}, counts[2] = {0, 0};
  int s = 0;
  if (N > unsigned(kSelectChunk)) {
    unsigned slots = nchunks;  // stage 0: raw chunks
    plan->nwg[0] = slots;
    plan->nin[0] = N;
    pairs[0] = size_t(R) * slots * cap * 8 /* (key, index) */;
    counts[0] = size_t(R) * slots * sizeof(unsigned);
    s = 1;
    while (slots > plan->group) {
      if (s == kSelectMaxStages) return false;
      const unsigned nwg = (slots + plan->group - 1) / plan->group;
      plan->nin[s] = slots;
      plan->nwg[s] = nwg;
      pairs[s & 1] = std::max(pairs[s & 1], size_t(R) * nwg * cap * 8 /* (key, index) */);
      counts[s & 1] = std::max(counts[s & 1], size_t(R) * nwg * sizeof(unsigned));
      slots = nwg;
      ++s;
    }
    plan->final_in = slots;
  } else {
    plan->final_in = N;
  }
  plan->stages = s;
  size_t off = ctl;
  for (int b = 0; b < 2; ++b) {
    plan->pair_off[b] = off;
    off += up(pairs[b]);
    plan->count_off[b] = off;
    off += up(counts[b]);
  }
  plan->total = off;
  return true;
}


onela_status_t check_select(int R, int prev_width, int vocab, int width, SelectPlan* plan) {
  if (R < 1 || R > 65536 || prev_width < 1 || vocab < 1 || width < 1) return ONELA_EINVAL;
  const uint64_t n = uint64_t(prev_width) * uint64_t(vocab);
  if (n > kSelectMaxCandidates || !select_plan(R, unsigned(n), unsigned(width), plan))
    return ONELA_EINVAL;
  return ONELA_OK;
}

// ---- per-step protocol --------------------------------------------------------
// resolve(t) -> append(t) -> decode(t) (decode may repeat), or fused(t); the
// next step starts only after the previous one was appended.

onela_status_t check_resolve(const Shape& s, const Protocol& pr, int step, int width,
                             const void* parents, const void* gather_out) {
  if (step != pr.resolved + 1 || pr.appended != pr.resolved) return ONELA_ESTEP;
  if (step >= s.tmax) return ONELA_ECAPACITY;
  if (width < 1 || width > s.wmax) return ONELA_ECAPACITY;
  if (step == 0 && parents) return ONELA_EINVAL;
  if (step > 0 && (!parents || !aligned4(parents))) return ONELA_EINVAL;
  if (gather_out && !aligned4(gather_out)) return ONELA_EINVAL;
  return ONELA_OK;
}

onela_status_t check_append(const Protocol& pr, int step, const void* k, const void* v,
                            const void* alpha, const void* beta) {
  if (step < 0 || step != pr.resolved || step != pr.appended + 1) return ONELA_ESTEP;
  if (!k || !v || !alpha || !beta) return ONELA_EINVAL;
  if (!aligned16(k) || !aligned16(v) || !aligned4(alpha) || !aligned4(beta))
    return ONELA_EINVAL;
  return ONELA_OK;
}

onela_status_t check_decode(const Protocol& pr, int step, const void* q, const void* o) {
  if (step < 0 || step != pr.resolved || step != pr.appended) return ONELA_ESTEP;
  if (!q || !o || !aligned16(q) || !aligned16(o)) return ONELA_EINVAL;
  return ONELA_OK;
}

onela_status_t check_fused(const Shape& s, const Protocol& pr, int step, int width,
                           const void* parents, const void* k, const void* v,
                           const void* alpha, const void* beta, const void* q,
                           const void* o, const void* gather_out) {
  const onela_status_t rc = check_resolve(s, pr, step, width, parents, gather_out);
  if (rc != ONELA_OK) return rc;
  if (!k || !v || !alpha || !beta || !q || !o) return ONELA_EINVAL;
  if (!aligned16(k) || !aligned16(v) || !aligned4(alpha) || !aligned4(beta) || !aligned16(q) ||
      !aligned16(o))
    return ONELA_EINVAL;
  return ONELA_OK;
}

}  // namespace onela
