// Internal declarations shared by the host side (onela_api.cpp) and the HIP
// kernels of libonela.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "host_plan.h"

namespace onela {

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


// ---- chunked prefill --------------------------------------------------------
hipError_t launch_prefill_chunked(const Shape& s, int prompt_len, const void* k, const void* v,
                                  const float* alpha, const float* beta, float* s0_out,
                                  void* workspace, hipStream_t st);

// ---- global top-W beam selection ------------------------------------------
// Device address of the allocation-free entry point's scratch array on the
// current device.
hipError_t select_scratch(void** out);
hipError_t launch_select(const SelectPlan& plan, int R, int prev_width, int vocab, int width,
                         const float* logp, const float* beam, int* parents, int* tokens,
                         float* scores, void* workspace, hipStream_t st);

}  // namespace onela
