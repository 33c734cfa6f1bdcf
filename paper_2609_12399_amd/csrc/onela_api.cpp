// Host side of libonela: argument validation, workspace carving, per-step
// protocol bookkeeping and kernel launches.  Every check that can fail runs
// before anything is enqueued, so a rejected call leaves no device work and
// no change in the context.
#include <atomic>
#include <cstdint>
#include <cstdlib>
#include <new>

#include "../../include/onela.h"
#include "internal.h"

using onela::aligned16;
using onela::aligned4;
using onela::Arena;
using onela::Layout;
using onela::Protocol;
using onela::Shape;
using onela::shape_of;

struct onela_ctx_s {
  Shape shape;
  Arena arena;
  hipStream_t stream;
  Protocol pr;  // steps resolved / appended, widths, status-word state
};

namespace {

bool launch_ok(hipError_t e) { return e == hipSuccess; }

// Registers the caller's buffers as step t's record slab (borrowed records).
void borrow_step(onela_ctx_s* c, int t, const void* k, const void* v, const float* alpha,
                 const float* beta) {
  c->arena.bk[t] = k;
  c->arena.bv[t] = v;
  c->arena.balpha[t] = alpha;
  c->arena.bbeta[t] = beta;
  c->arena.bw[t] = c->pr.widths[t];
}

}  // namespace


extern "C" {

const char* onela_status_str(onela_status_t st) {
  switch (st) {
    case ONELA_OK: return "ok";
    case ONELA_EINVAL: return "invalid argument";
    case ONELA_ESTEP: return "call out of step order";
    case ONELA_EPARENT: return "parent index out of range (device)";
    case ONELA_ECAPACITY: return "capacity exceeded";
    case ONELA_EHIP: return "HIP runtime error";
    case ONELA_ENOMEM: return "host allocation failed";
  }
  return "unknown status";
}

onela_status_t onela_check_config(const onela_config_t* cfg) {
  Shape s;
  return shape_of(cfg, &s);
}

size_t onela_workspace_bytes(const onela_config_t* cfg) {
  Shape s;
  if (shape_of(cfg, &s) != ONELA_OK) return 0;
  return onela::layout_of(s).total;
}

namespace {
// Compute units of the current device, queried once per device (a host-side
// attribute query; nothing is enqueued).  0 if it cannot be read.
int device_compute_units() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v <= 0) {
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    cache[dev].store(v, std::memory_order_relaxed);
  }
  return v > 0 ? v : 0;
}
}  // namespace

onela_status_t onela_init(const onela_config_t* cfg, const float* s0,
                          void* workspace, size_t workspace_bytes, void* stream,
                          onela_ctx_t* out) {
  Shape s;
  onela_status_t rc = shape_of(cfg, &s);
  if (rc != ONELA_OK) return rc;
  if (!s0 || !workspace || !out || !aligned16(s0)) return ONELA_EINVAL;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0) return ONELA_EINVAL;
  const Layout l = onela::layout_of(s);
  if (workspace_bytes < l.total) return ONELA_ECAPACITY;
  s.cus = device_compute_units();

  onela_ctx_s* c = new (std::nothrow) onela_ctx_s();
  if (!c) return ONELA_ENOMEM;
  c->shape = s;
  c->stream = static_cast<hipStream_t>(stream);
  c->pr = Protocol{};
  char* p = static_cast<char*>(workspace);
  c->arena.status = reinterpret_cast<int*>(p);
  p += l.status;
  c->arena.anc[0] = reinterpret_cast<int*>(p);
  p += l.anc;
  c->arena.anc[1] = reinterpret_cast<int*>(p);
  p += l.anc;
  c->arena.s0 = s0;
  c->arena.s_frag = reinterpret_cast<uint16_t*>(p);
  p += l.s_frag;
  c->arena.k = s.borrow ? nullptr : p;
  p += l.k;
  c->arena.v = s.borrow ? nullptr : p;
  p += l.v;
  c->arena.ab = s.borrow ? nullptr : reinterpret_cast<float2*>(p);
  p += l.ab;
  c->arena.d = s.delta ? p : nullptr;
  p += l.d;
  c->arena.dsc = s.delta ? reinterpret_cast<unsigned*>(p) : nullptr;

  *out = c;
  return ONELA_OK;
}

onela_status_t onela_reset(onela_ctx_t c) {
  if (!c) return ONELA_EINVAL;
  c->pr.resolved = -1;
  c->pr.appended = -1;
  c->pr.search_zeroed = false;
  return ONELA_OK;
}

onela_status_t onela_resolve_ancestry(onela_ctx_t c, int32_t step, int32_t width,
                                      const int32_t* parents, int32_t* gather_out) {
  if (!c) return ONELA_EINVAL;
  const Shape& s = c->shape;
  Protocol& pr = c->pr;
  const onela_status_t rc = onela::check_resolve(s, pr, step, width, parents, gather_out);
  if (rc != ONELA_OK) return rc;
  if (step > 0) {
    // The step-0 decode launch zeroes the status word of a new search.  When
    // the caller resolves step 1 without having decoded step 0, zero it here
    // first, so that what the resolve kernel flags is not mixed with a word
    // that was never cleared (or still holds an earlier search's error).
    if (!pr.search_zeroed) {
      if (!launch_ok(onela::launch_clear_status(c->arena.status, c->stream))) return ONELA_EHIP;
      pr.search_zeroed = true;
      pr.status_live = true;
    }
    hipError_t e = onela::launch_resolve(s, step, width, pr.widths[step - 1], parents,
                                         c->arena.anc[(step - 1) & 1],
                                         c->arena.anc[step & 1], gather_out,
                                         c->arena.status, c->stream);
    if (!launch_ok(e)) return ONELA_EHIP;
  }
  pr.widths[step] = width;
  pr.resolved = step;
  return ONELA_OK;
}

onela_status_t onela_append_records(onela_ctx_t c, int32_t step, const void* k,
                                    const void* v, const float* alpha,
                                    const float* beta) {
  if (!c) return ONELA_EINVAL;
  const onela_status_t rc = onela::check_append(c->pr, step, k, v, alpha, beta);
  if (rc != ONELA_OK) return rc;
  if (c->shape.borrow) {
    borrow_step(c, step, k, v, alpha, beta);
  } else {
    hipError_t e = onela::launch_append(c->shape, step, c->pr.widths[step], k, v, alpha,
                                        beta, c->arena, c->stream);
    if (!launch_ok(e)) return ONELA_EHIP;
  }
  c->pr.appended = step;
  return ONELA_OK;
}

onela_status_t onela_decode_step(onela_ctx_t c, int32_t step, const void* q, float* o) {
  if (!c) return ONELA_EINVAL;
  const onela_status_t rc = onela::check_decode(c->pr, step, q, o);
  if (rc != ONELA_OK) return rc;
  const int width = c->pr.widths[step];
  hipError_t e = c->shape.delta
                     ? onela::launch_replay_decode(c->shape, step, width, q, o, c->arena,
                                                   c->stream)
                     : onela::launch_decode(c->shape, step, width, q, o, c->arena, c->stream);
  if (!launch_ok(e)) return ONELA_EHIP;
  if (step == 0) c->pr.status_live = c->pr.search_zeroed = true;
  return ONELA_OK;
}

onela_status_t onela_decode_step_fused(onela_ctx_t c, int32_t step, int32_t width,
                                       const int32_t* parents, const void* k, const void* v,
                                       const float* alpha, const float* beta, const void* q,
                                       float* o, int32_t* gather_out) {
  if (!c) return ONELA_EINVAL;
  const Shape& s = c->shape;
  Protocol& pr = c->pr;
  const onela_status_t rc =
      onela::check_fused(s, pr, step, width, parents, k, v, alpha, beta, q, o, gather_out);
  if (rc != ONELA_OK) return rc;
  const int prev = step > 0 ? pr.widths[step - 1] : 0;
  hipError_t e = s.delta ? onela::launch_replay_fused(s, step, width, prev, parents, k, v, alpha,
                                                      beta, q, o, gather_out, c->arena, c->stream)
                         : onela::launch_fused_step(s, step, width, prev, parents, k, v, alpha,
                                                    beta, q, o, gather_out, c->arena, c->stream);
  if (!launch_ok(e)) return ONELA_EHIP;
  pr.widths[step] = width;
  if (s.borrow) borrow_step(c, step, k, v, alpha, beta);
  pr.resolved = step;
  pr.appended = step;
  if (step == 0) pr.status_live = pr.search_zeroed = true;
  return ONELA_OK;
}

onela_status_t onela_get_device_status(onela_ctx_t c) {
  if (!c) return ONELA_EINVAL;
  if (hipStreamSynchronize(c->stream) != hipSuccess) return ONELA_EHIP;
  if (!c->pr.status_live) return ONELA_OK;  // no step has run: nothing was flagged
  int word = 0;
  if (hipMemcpy(&word, c->arena.status, sizeof(int), hipMemcpyDeviceToHost) != hipSuccess)
    return ONELA_EHIP;
  if (word == 0) return ONELA_OK;
  if (!launch_ok(onela::launch_clear_status(c->arena.status, c->stream)) ||
      hipStreamSynchronize(c->stream) != hipSuccess)
    return ONELA_EHIP;
  return ONELA_EPARENT;
}

void onela_destroy(onela_ctx_t c) { delete c; }

onela_status_t onela_prefill_state(const onela_config_t* cfg, int32_t prompt_len,
                                   const void* k, const void* v, const float* alpha,
                                   const float* beta, float* s0_out, void* stream) {
  Shape s;
  onela_status_t rc = shape_of(cfg, &s);
  if (rc != ONELA_OK) return rc;
  if (prompt_len < 0 || !s0_out || !aligned16(s0_out)) return ONELA_EINVAL;
  if (prompt_len > 0 && (!k || !v || !alpha || !beta || !aligned16(k) || !aligned16(v) ||
                         !aligned4(alpha) || !aligned4(beta)))
    return ONELA_EINVAL;
  hipError_t e = onela::launch_prefill(s, prompt_len, k, v, alpha, beta, s0_out,
                                       static_cast<hipStream_t>(stream));
  return launch_ok(e) ? ONELA_OK : ONELA_EHIP;
}

size_t onela_prefill_workspace_bytes(const onela_config_t* cfg, int32_t prompt_len) {
  Shape s;
  if (shape_of(cfg, &s) != ONELA_OK || prompt_len < 0) return 0;
  return onela::prefill_chunked_workspace_bytes(s, prompt_len);
}

onela_status_t onela_prefill_state_chunked(const onela_config_t* cfg, int32_t prompt_len,
                                           const void* k, const void* v, const float* alpha,
                                           const float* beta, float* s0_out, void* workspace,
                                           size_t workspace_bytes, void* stream) {
  Shape s;
  const onela_status_t rc = shape_of(cfg, &s);
  if (rc != ONELA_OK) return rc;
  if (prompt_len < 0 || !s0_out || !aligned16(s0_out)) return ONELA_EINVAL;
  if (prompt_len > 0 && (!k || !v || !alpha || !beta || !aligned16(k) || !aligned16(v) ||
                         !aligned4(alpha) || !aligned4(beta)))
    return ONELA_EINVAL;
  const size_t need = onela::prefill_chunked_workspace_bytes(s, prompt_len);
  if (need > 0 && (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0))
    return ONELA_EINVAL;
  if (workspace_bytes < need) return ONELA_ECAPACITY;
  const hipError_t e =
      onela::launch_prefill_chunked(s, prompt_len, k, v, alpha, beta, s0_out, workspace,
                                    static_cast<hipStream_t>(stream));
  return launch_ok(e) ? ONELA_OK : ONELA_EHIP;
}

size_t onela_fullstate_workspace_bytes(const onela_config_t* cfg) {
  Shape s;
  if (shape_of(cfg, &s) != ONELA_OK) return 0;
  return 2 * sizeof(float) * size_t(s.R) * s.wmax * s.HV * size_t(s.dv) * s.dk;
}

onela_status_t onela_fullstate_step(const onela_config_t* cfg, int32_t step,
                                    int32_t width, int32_t prev_width,
                                    const int32_t* parents, const float* s0,
                                    const void* q, const void* k, const void* v,
                                    const float* alpha, const float* beta, float* o,
                                    void* workspace, size_t workspace_bytes,
                                    int32_t* status_word, void* stream) {
  Shape s;
  onela_status_t rc = shape_of(cfg, &s);
  if (rc != ONELA_OK) return rc;
  if (step < 0 || width < 1 || width > s.wmax) return ONELA_ECAPACITY;
  if (step > 0 && (prev_width < 1 || prev_width > s.wmax)) return ONELA_ECAPACITY;
  if (step == 0 && parents) return ONELA_EINVAL;
  if (step > 0 && (!parents || !aligned4(parents))) return ONELA_EINVAL;
  if (!s0 || !q || !k || !v || !alpha || !beta || !o || !workspace) return ONELA_EINVAL;
  if (!aligned16(s0) || !aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) ||
      !aligned4(alpha) || !aligned4(beta) || !aligned16(workspace))
    return ONELA_EINVAL;
  if (status_word && !aligned4(status_word)) return ONELA_EINVAL;
  const size_t half = sizeof(float) * size_t(s.R) * s.wmax * s.HV * size_t(s.dv) * s.dk;
  if (workspace_bytes < 2 * half) return ONELA_ECAPACITY;
  float* base = static_cast<float*>(workspace);
  float* buf[2] = {base, base + half / sizeof(float)};
  hipError_t e = onela::launch_fullstate(s, step, width, prev_width, parents, s0, q, k, v,
                                         alpha, beta, o, buf[(step + 1) & 1], buf[step & 1],
                                         status_word, static_cast<hipStream_t>(stream));
  return launch_ok(e) ? ONELA_OK : ONELA_EHIP;
}

uint64_t onela_capacity_bytes(int32_t R, int32_t HV, int32_t dk, int32_t dv, int32_t beams,
                              int32_t steps, int32_t state_bytes, int32_t record_bytes) {
  if (R < 0 || HV < 0 || dk < 0 || dv < 0 || beams < 0 || steps < 0 || state_bytes < 0 ||
      record_bytes < 0)
    return 0;
  const uint64_t ctx = uint64_t(R) * HV * uint64_t(dv) * dk * state_bytes;
  const uint64_t rec = uint64_t(steps) * R * uint64_t(beams) * HV * record_bytes;
  return ctx + rec;
}

uint64_t onela_fullstate_capacity_bytes(int32_t R, int32_t HV, int32_t dk, int32_t dv,
                                        int32_t beams, int32_t state_bytes) {
  if (R < 0 || HV < 0 || dk < 0 || dv < 0 || beams < 0 || state_bytes < 0) return 0;
  return uint64_t(R) * beams * HV * uint64_t(dv) * dk * state_bytes;
}

onela_status_t onela_select_workspace_bytes(int32_t num_requests, int32_t prev_width,
                                            int32_t vocab, int32_t width, size_t* bytes) {
  if (!bytes) return ONELA_EINVAL;
  *bytes = 0;
  onela::SelectPlan plan;
  const onela_status_t rc = onela::check_select(num_requests, prev_width, vocab, width, &plan);
  if (rc != ONELA_OK) return rc;
  *bytes = plan.total;
  return ONELA_OK;
}

onela_status_t onela_select_beams(int32_t num_requests, int32_t prev_width, int32_t vocab,
                                  int32_t width, const float* logp, const float* beam_scores,
                                  int32_t* parents_out, int32_t* tokens_out, float* scores_out,
                                  void* workspace, size_t workspace_bytes, void* stream) {
  size_t need = 0;
  const onela_status_t st =
      onela_select_workspace_bytes(num_requests, prev_width, vocab, width, &need);
  if (st != ONELA_OK) return st;
  if (!logp || !parents_out || !tokens_out || !scores_out || !aligned4(logp) ||
      !aligned4(parents_out) || !aligned4(tokens_out) || !aligned4(scores_out))
    return ONELA_EINVAL;
  if (beam_scores && !aligned4(beam_scores)) return ONELA_EINVAL;
  if (need > 0 && (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0))
    return ONELA_EINVAL;
  if (workspace_bytes < need) return ONELA_ECAPACITY;
  onela::SelectPlan plan;
  onela::select_plan(num_requests, unsigned(prev_width) * unsigned(vocab), unsigned(width),
                     &plan);
  const hipError_t e = onela::launch_select(plan, num_requests, prev_width, vocab, width, logp,
                                            beam_scores, parents_out, tokens_out, scores_out,
                                            workspace, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ONELA_OK : ONELA_EHIP;
}

onela_status_t onela_select_beams_noalloc(int32_t num_requests, int32_t prev_width,
                                          int32_t vocab, int32_t width, const float* logp,
                                          const float* beam_scores, int32_t* parents_out,
                                          int32_t* tokens_out, float* scores_out,
                                          void* stream) {
  size_t need = 0;
  const onela_status_t st =
      onela_select_workspace_bytes(num_requests, prev_width, vocab, width, &need);
  if (st != ONELA_OK) return st;
  if (need > onela::kSelectScratchBytes) return ONELA_ECAPACITY;
  if (!logp || !parents_out || !tokens_out || !scores_out || !aligned4(logp) ||
      !aligned4(parents_out) || !aligned4(tokens_out) || !aligned4(scores_out))
    return ONELA_EINVAL;
  if (beam_scores && !aligned4(beam_scores)) return ONELA_EINVAL;
  void* ws = nullptr;
  if (onela::select_scratch(&ws) != hipSuccess) return ONELA_EHIP;
  onela::SelectPlan plan;
  onela::select_plan(num_requests, unsigned(prev_width) * unsigned(vocab), unsigned(width),
                     &plan);
  const hipError_t e = onela::launch_select(plan, num_requests, prev_width, vocab, width, logp,
                                            beam_scores, parents_out, tokens_out, scores_out,
                                            ws, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ONELA_OK : ONELA_EHIP;
}

}  // extern "C"
