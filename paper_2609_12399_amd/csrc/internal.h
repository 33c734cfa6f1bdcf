// Internal declarations shared by the host side (onela_api.cpp) and the HIP
// kernels of libonela.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

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

// Device views carved out of the caller's workspace.
struct Arena {
  int* status;       // sticky error bits
  int* anc[2];       // ancestry h_t, [R][wmax][tmax] int32, buffer t % 2
  const float* s0;   // S_ctx fp32 [R][HV][dv][dk], borrowed from the caller
  uint16_t* s_frag;  // S_ctx as bf16 hi/lo in MFMA A-fragment order (from step 0)
  void* k;           // [R][tmax][HK][wmax][dk] io dtype
  void* v;           // [R][tmax][HV][wmax][dv] io dtype
  float2* ab;        // [R][tmax][HV][wmax] (alpha, beta)
  void* d;           // delta records [R][tmax][HV][wmax][dv], fp16 (bf16 io) / fp32; or null
  unsigned* dsc;     // per delta row: one int8 scale exponent per row slice [R][tmax][HV][wmax]
  // borrowed records (Shape::borrow): the caller's buffers of step j,
  // k [R][w[j]][HK][dk], v [R][w[j]][HV][dv], alpha / beta [R][w[j]][HV]
  const void* bk[kMaxSteps];
  const void* bv[kMaxSteps];
  const float* balpha[kMaxSteps];
  const float* bbeta[kMaxSteps];
  int bw[kMaxSteps];
};

// Bytes of each region, in workspace order, each rounded up to 256.
struct Layout {
  size_t status, anc, s_frag, k, v, ab, d, ds, total;
};
Layout layout_of(const Shape& s);

// ---- launchers (each returns hipGetLastError() after the launch) ---------
hipError_t launch_clear_status(int* status, hipStream_t st);
hipError_t launch_resolve(const Shape& s, int step, int width, int prev_width,
                          const int* parents, const int* anc_prev, int* anc_cur,
                          int* gather_out, int* status, hipStream_t st);
hipError_t launch_append(const Shape& s, int step, int width, const void* k,
                         const void* v, const float* alpha, const float* beta,
                         const Arena& a, hipStream_t st);
hipError_t launch_decode(const Shape& s, int step, int width, const void* q,
                         float* o, const Arena& a, hipStream_t st);
hipError_t launch_fused_step(const Shape& s, int step, int width, int prev_width,
                             const int* parents, const void* k, const void* v,
                             const float* alpha, const float* beta, const void* q, float* o,
                             int* gather_out, const Arena& a, hipStream_t st);
hipError_t launch_replay_decode(const Shape& s, int step, int width, const void* q, float* o,
                                const Arena& a, hipStream_t st);
hipError_t launch_replay_fused(const Shape& s, int step, int width, int prev_width,
                               const int* parents, const void* k, const void* v,
                               const float* alpha, const float* beta, const void* q, float* o,
                               int* gather_out, const Arena& a, hipStream_t st);
hipError_t launch_prefill(const Shape& s, int prompt_len, const void* k,
                          const void* v, const float* alpha, const float* beta,
                          float* s0_out, hipStream_t st);
hipError_t launch_fullstate(const Shape& s, int step, int width, int prev_width,
                            const int* parents, const float* s0, const void* q,
                            const void* k, const void* v, const float* alpha,
                            const float* beta, float* o, const float* states_in,
                            float* states_out, int* status, hipStream_t st);

// True when the decode kernel has an instance for this shape.
bool decode_supported(const Shape& s);

// ---- chunked prefill --------------------------------------------------------
constexpr int kPrefillChunk = 64;  // tokens per chunk
size_t prefill_chunked_workspace_bytes(const Shape& s, int prompt_len);
hipError_t launch_prefill_chunked(const Shape& s, int prompt_len, const void* k, const void* v,
                                  const float* alpha, const float* beta, float* s0_out,
                                  void* workspace, hipStream_t st);

// ---- global top-W beam selection ------------------------------------------
constexpr int kSelectThreads = 512;            // one workgroup
constexpr int kSelectChunk = 16384;            // candidates per workgroup
constexpr int kSelectMaxWidth = 4096;          // W kept per request
constexpr int kSelectMaxStages = 16;           // reduction stages before the final one
constexpr unsigned kSelectMaxCandidates = 1u << 29;  // W_prev * V per request
constexpr int kSelectMaxGatherSlots = 2048;          // chunks per request, two-pass path
constexpr int kSelectOnePassMaxRequests = 64;        // requests of a one-pass call
constexpr size_t kSelectCtlBytes = 1024;             // one-pass control block, workspace start

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
  // Two-pass path (see kernels_select.hip): per request nseg wave maxima,
  // then nchunks slots of `cap` pairs and their counts.
  bool two_pass;
  unsigned nchunks, nseg;
  size_t seg_off, slot_off, cnt_off;
};
bool select_plan(int R, unsigned N, unsigned W, SelectPlan* plan);
// Size of the per-device scratch array of the allocation-free selection
// entry point, and its device address on the current device.
constexpr size_t kSelectScratchBytes = size_t(32) << 20;
hipError_t select_scratch(void** out);
hipError_t launch_select(const SelectPlan& plan, int R, int prev_width, int vocab, int width,
                         const float* logp, const float* beam, int* parents, int* tokens,
                         float* scores, void* workspace, hipStream_t st);

}  // namespace onela
