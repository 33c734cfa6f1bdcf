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

using onela::Arena;
using onela::Layout;
using onela::Shape;

struct onela_ctx_s {
  Shape shape;
  Arena arena;
  hipStream_t stream;
  int resolved;  // last step whose ancestry was resolved (-1: none)
  bool status_live;  // a launch that zeroes the status word was enqueued (ever)
  bool search_zeroed;  // ... in the current beam search (since init / reset)
  int appended;  // last step whose records were appended (-1: none)
  int widths[onela::kMaxSteps];
};

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

size_t round256(size_t x) { return (x + 255) & ~size_t(255); }

onela_status_t shape_of(const onela_config_t* c, Shape* s) {
  if (!c) return ONELA_EINVAL;
  if (c->num_requests < 1 || c->num_qk_heads < 1 || c->num_v_heads < 1)
    return ONELA_EINVAL;
  if (c->num_v_heads % c->num_qk_heads) return ONELA_EINVAL;
  if (c->max_beams < 1 || c->max_beams > 65536) return ONELA_EINVAL;
  if (c->max_steps < 1 || c->max_steps > onela::kMaxSteps) return ONELA_EINVAL;
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
  if (!onela::decode_supported(t)) return ONELA_EINVAL;
  // the kernels form 32-bit byte offsets: every region must stay below 2 GiB
  const double big = double(t.R) * t.tmax * (t.HV > t.HK ? t.HV : t.HK) * t.wmax *
                     (t.dv > t.dk ? t.dv : t.dk) * t.io_bytes();
  const double outb = double(t.R) * t.wmax * t.HV * t.dv * 4.0;
  const double s0b = double(t.R) * t.HV * t.dv * t.dk * 4.0;
  if (big >= 2147483648.0 || outb >= 2147483648.0 || s0b >= 2147483648.0) return ONELA_EINVAL;
  *s = t;
  return ONELA_OK;
}

bool launch_ok(hipError_t e) { return e == hipSuccess; }

// Registers the caller's buffers as step t's record slab (borrowed records).
void borrow_step(onela_ctx_s* c, int t, const void* k, const void* v, const float* alpha,
                 const float* beta) {
  c->arena.bk[t] = k;
  c->arena.bv[t] = v;
  c->arena.balpha[t] = alpha;
  c->arena.bbeta[t] = beta;
  c->arena.bw[t] = c->widths[t];
}

}  // namespace

namespace onela {

Layout layout_of(const Shape& s) {
  Layout l{};
  const size_t R = s.R, T = s.tmax, W = s.wmax;
  l.status = 256;
  l.anc = round256(sizeof(int) * R * W * T);
  l.s_frag = round256(sizeof(uint16_t) * 2 * R * s.HV * size_t(s.dv) * s.dk);
  const size_t arena = s.borrow ? 0 : 1;  // borrowed records need no arena
  l.k = arena * round256(size_t(s.io_bytes()) * R * T * s.HK * W * s.dk);
  l.v = arena * round256(size_t(s.io_bytes()) * R * T * s.HV * W * s.dv);
  l.ab = arena * round256(sizeof(float2) * R * T * s.HV * W);
  l.d = s.delta ? l.v : 0;  // delta rows take the size of input v rows (fp16 / fp32)
  l.ds = s.delta ? round256(sizeof(unsigned) * R * T * s.HV * W) : 0;  // delta row scales
  l.total = l.status + 2 * l.anc + l.s_frag + l.k + l.v + l.ab + l.d + l.ds;
  return l;
}

}  // namespace onela

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
  c->resolved = -1;
  c->appended = -1;
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

  c->status_live = false;
  c->search_zeroed = false;
  *out = c;
  return ONELA_OK;
}

onela_status_t onela_reset(onela_ctx_t c) {
  if (!c) return ONELA_EINVAL;
  c->resolved = -1;
  c->appended = -1;
  c->search_zeroed = false;
  return ONELA_OK;
}

onela_status_t onela_resolve_ancestry(onela_ctx_t c, int32_t step, int32_t width,
                                      const int32_t* parents, int32_t* gather_out) {
  if (!c) return ONELA_EINVAL;
  const Shape& s = c->shape;
  if (step != c->resolved + 1 || c->appended != c->resolved) return ONELA_ESTEP;
  if (step >= s.tmax) return ONELA_ECAPACITY;
  if (width < 1 || width > s.wmax) return ONELA_ECAPACITY;
  if (step == 0 && parents) return ONELA_EINVAL;
  if (step > 0 && (!parents || !aligned4(parents))) return ONELA_EINVAL;
  if (gather_out && !aligned4(gather_out)) return ONELA_EINVAL;
  if (step > 0) {
    // The step-0 decode launch zeroes the status word of a new search.  When
    // the caller resolves step 1 without having decoded step 0, zero it here
    // first, so that what the resolve kernel flags is not mixed with a word
    // that was never cleared (or still holds an earlier search's error).
    if (!c->search_zeroed) {
      if (!launch_ok(onela::launch_clear_status(c->arena.status, c->stream))) return ONELA_EHIP;
      c->search_zeroed = true;
      c->status_live = true;
    }
    hipError_t e = onela::launch_resolve(s, step, width, c->widths[step - 1], parents,
                                         c->arena.anc[(step - 1) & 1],
                                         c->arena.anc[step & 1], gather_out,
                                         c->arena.status, c->stream);
    if (!launch_ok(e)) return ONELA_EHIP;
  }
  c->widths[step] = width;
  c->resolved = step;
  return ONELA_OK;
}

onela_status_t onela_append_records(onela_ctx_t c, int32_t step, const void* k,
                                    const void* v, const float* alpha,
                                    const float* beta) {
  if (!c) return ONELA_EINVAL;
  if (step != c->resolved || step != c->appended + 1) return ONELA_ESTEP;
  if (!k || !v || !alpha || !beta) return ONELA_EINVAL;
  if (!aligned16(k) || !aligned16(v) || !aligned4(alpha) || !aligned4(beta))
    return ONELA_EINVAL;
  if (c->shape.borrow) {
    borrow_step(c, step, k, v, alpha, beta);
  } else {
    hipError_t e = onela::launch_append(c->shape, step, c->widths[step], k, v, alpha,
                                        beta, c->arena, c->stream);
    if (!launch_ok(e)) return ONELA_EHIP;
  }
  c->appended = step;
  return ONELA_OK;
}

onela_status_t onela_decode_step(onela_ctx_t c, int32_t step, const void* q, float* o) {
  if (!c) return ONELA_EINVAL;
  if (step < 0 || step != c->resolved || step != c->appended) return ONELA_ESTEP;
  if (!q || !o || !aligned16(q) || !aligned16(o)) return ONELA_EINVAL;
  hipError_t e = c->shape.delta
                     ? onela::launch_replay_decode(c->shape, step, c->widths[step], q, o,
                                                   c->arena, c->stream)
                     : onela::launch_decode(c->shape, step, c->widths[step], q, o, c->arena,
                                            c->stream);
  if (!launch_ok(e)) return ONELA_EHIP;
  if (step == 0) c->status_live = c->search_zeroed = true;
  return ONELA_OK;
}

onela_status_t onela_decode_step_fused(onela_ctx_t c, int32_t step, int32_t width,
                                       const int32_t* parents, const void* k, const void* v,
                                       const float* alpha, const float* beta, const void* q,
                                       float* o, int32_t* gather_out) {
  if (!c) return ONELA_EINVAL;
  const Shape& s = c->shape;
  if (step != c->resolved + 1 || c->appended != c->resolved) return ONELA_ESTEP;
  if (step >= s.tmax) return ONELA_ECAPACITY;
  if (width < 1 || width > s.wmax) return ONELA_ECAPACITY;
  if (step == 0 && parents) return ONELA_EINVAL;
  if (step > 0 && (!parents || !aligned4(parents))) return ONELA_EINVAL;
  if (gather_out && !aligned4(gather_out)) return ONELA_EINVAL;
  if (!k || !v || !alpha || !beta || !q || !o) return ONELA_EINVAL;
  if (!aligned16(k) || !aligned16(v) || !aligned4(alpha) || !aligned4(beta) || !aligned16(q) ||
      !aligned16(o))
    return ONELA_EINVAL;
  const int prev = step > 0 ? c->widths[step - 1] : 0;
  hipError_t e = s.delta ? onela::launch_replay_fused(s, step, width, prev, parents, k, v, alpha,
                                                      beta, q, o, gather_out, c->arena, c->stream)
                         : onela::launch_fused_step(s, step, width, prev, parents, k, v, alpha,
                                                    beta, q, o, gather_out, c->arena, c->stream);
  if (!launch_ok(e)) return ONELA_EHIP;
  c->widths[step] = width;
  if (s.borrow) borrow_step(c, step, k, v, alpha, beta);
  c->resolved = step;
  c->appended = step;
  if (step == 0) c->status_live = c->search_zeroed = true;
  return ONELA_OK;
}

onela_status_t onela_get_device_status(onela_ctx_t c) {
  if (!c) return ONELA_EINVAL;
  if (hipStreamSynchronize(c->stream) != hipSuccess) return ONELA_EHIP;
  if (!c->status_live) return ONELA_OK;  // no step has run: nothing was flagged
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
  if (num_requests < 1 || num_requests > 65536 || prev_width < 1 || vocab < 1 || width < 1)
    return ONELA_EINVAL;
  const uint64_t n = uint64_t(prev_width) * uint64_t(vocab);
  if (n > onela::kSelectMaxCandidates ||
      !onela::select_plan(num_requests, unsigned(n), unsigned(width), &plan))
    return ONELA_EINVAL;
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
