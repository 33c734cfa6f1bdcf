// Host-side plans and checks of libonela: shapes, workspace layouts, the
// beam-selection launch plan and the per-step protocol.  Plain C++ with no
// HIP dependency, so that it is built and run under the host sanitizers as
// well as into the library.  Not part of the public ABI.
#pragma once

#include <cstddef>
#include <cstdint>

#include "../../include/onela.h"

namespace onela {


// Maximum records in one beam's chain (decode steps 0 .. kMaxSteps-1).
constexpr int kMaxSteps = 8;
// Ancestry entries (previous beams x steps <= t-2) a fused decode step at
// t >= 2 stages in LDS; larger tables are read row by row from global memory.
constexpr int kAncTable = 2048;
// The staged table's limit from chains of 5 records on (t >= 4).
constexpr int kAncTableLong = 1024;

// Decode tiling: 16-beam MFMA column blocks per workgroup.
constexpr int kDecodeBeamBlocks = 2;

// Bits of the sticky device status word.
constexpr int kStatusParent = 1;

struct Shape {
  int R, HK, HV, dk, dv;
  int wmax, tmax;
  bool bf16;  // q/k/v stored as bf16 bits (else fp32)
  bool delta;  // records are (alpha, delta, k) transition records (else step inputs)
  bool borrow;  // step-input records stay in the caller's buffers (no arena copy)
  int cus = 0;  // compute units of the context's device (0: not known)
  int io_bytes() const { return bf16 ? 2 : 4; }
};


// Bytes of each region, in workspace order, each rounded up to 256.
struct Layout {
  size_t status, anc, s_frag, k, v, ab, d, ds, total;
};
Layout layout_of(const Shape& s);

// True when the decode kernel has an instance for this shape.
bool decode_supported(const Shape& s);

// Tokens per chunk of the chunked prefill and its workspace size.
constexpr int kPrefillChunk = 64;  // tokens per chunk
size_t prefill_chunked_workspace_bytes(const Shape& s, int prompt_len);

// ---- global top-W beam selection ------------------------------------------
constexpr int kSelectThreads = 512;            // one workgroup
constexpr int kSelectChunk = 16384;            // candidates per workgroup
constexpr int kSelectMaxWidth = 4096;          // W kept per request
constexpr int kSelectMaxStages = 16;           // reduction stages before the final one
constexpr unsigned kSelectMaxCandidates = 1u << 29;  // W_prev * V per request
constexpr int kSelectMaxGatherSlots = 2048;          // chunks per request, two-pass path
constexpr int kSelectOnePassMaxRequests = 64;        // requests of a one-pass call
constexpr size_t kSelectCtlBytes = 1024;             // one-pass control block, workspace start
// One-pass wave summaries (16 bytes each, at most 8192: R * nchunks <= 1024),
// right after the control block; no other path writes this region.
constexpr size_t kSelectSummaryBytes = size_t(8192) * 16;

// Launch plan (tree path).  Stage 0 reads the raw scores in nwg[0] chunks of
// kSelectChunk per request; stage s >= 1 reads the nin[s] output slots of
// stage s - 1, `group` slots per workgroup.  Every stage workgroup writes one
// slot of `cap` (key, index) pairs plus a count into buffer s % 2 of the
// workspace.  The final launch reads final_in slots (or, with no stage, the
// final_in raw scores) per request.
struct SelectPlan {
  int stages;
  unsigned nin[kSelectMaxStages], nwg[kSelectMaxStages];
  unsigned final_in;
  unsigned cap, group;
  size_t pair_off[2], count_off[2], total;
  // Two-pass and one-pass paths (see kernels_select.hip): per request nseg
  // wave summaries or maxima (two-pass; the one-pass summaries have their own
  // region), one bound word, then nchunks slots of `cap` pairs and their
  // counts.
  bool two_pass;
  unsigned nchunks, nseg;
  size_t seg_off, bound_off, slot_off, cnt_off;
};
bool select_plan(int R, unsigned N, unsigned W, SelectPlan* plan);
// Size of the per-device scratch array of the allocation-free selection
// entry point.
constexpr size_t kSelectScratchBytes = size_t(32) << 20;

// ---- validation and the per-step protocol -----------------------------------

// The Shape of a configuration, or ONELA_EINVAL.
onela_status_t shape_of(const onela_config_t* cfg, Shape* out);

// Per-context protocol state: the last step resolved and appended (-1:
// none), the width of every resolved step, and whether the status word has
// been zeroed (ever / in the current beam search).
struct Protocol {
  int resolved = -1;
  int appended = -1;
  int widths[kMaxSteps] = {};
  bool status_live = false;
  bool search_zeroed = false;
};

// Checks of each entry point's arguments against the shape and the protocol
// state (no side effect); ONELA_OK when the call may proceed.
onela_status_t check_resolve(const Shape& s, const Protocol& pr, int step, int width,
                             const void* parents, const void* gather_out);
onela_status_t check_append(const Protocol& pr, int step, const void* k, const void* v,
                            const void* alpha, const void* beta);
onela_status_t check_decode(const Protocol& pr, int step, const void* q, const void* o);
onela_status_t check_fused(const Shape& s, const Protocol& pr, int step, int width,
                           const void* parents, const void* k, const void* v,
                           const void* alpha, const void* beta, const void* q,
                           const void* o, const void* gather_out);
// The selection plan of a call, or ONELA_EINVAL.
onela_status_t check_select(int R, int prev_width, int vocab, int width, SelectPlan* plan);

bool aligned16(const void* p);
bool aligned4(const void* p);

}  // namespace onela
