// Record store and ancestry index kernels (gfx950).
//
//   clear_status  zero the sticky device status word
//   resolve       ancestry index update, Sec. 3.3 Eq. 5 (integer, exact)
//   append        records of one step -> head-major arena slab (Sec. 3.3:
//                 written once into the current step's slots, never moved)
#include "internal.h"

namespace onela {
namespace {

__global__ void clear_status_kernel(int* status) {
  if (threadIdx.x == 0) status[0] = 0;
}

// Eq. 5: h_t(b, j) = h_{t-1}(pi_t(b), j) for j < t-1, h_t(b, t-1) = pi_t(b).
// One thread per (request, beam).  An out-of-range parent writes -1 into
// every index of that beam and raises the sticky status bit.
__global__ void resolve_kernel(const int* __restrict__ parents, const int* __restrict__ anc_prev,
                               int* __restrict__ anc_cur, int* __restrict__ gather_out,
                               int* __restrict__ status, int R, int width, int prev_width,
                               int wmax, int tmax, int step) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= R * width) return;
  const int r = i / width, b = i - r * width;
  const int par = parents[i];
  const bool ok = par >= 0 && par < prev_width;
  int* dst = anc_cur + (long(r) * wmax + b) * tmax;
  int* g = gather_out ? gather_out + long(i) * step : nullptr;
  if (!ok) {
    atomicOr(status, kStatusParent);
    for (int j = 0; j < step; ++j) {
      dst[j] = -1;
      if (g) g[j] = -1;
    }
    return;
  }
  const int* src = anc_prev + (long(r) * wmax + par) * tmax;
  for (int j = 0; j < step - 1; ++j) {
    const int h = src[j];
    dst[j] = h;
    if (g) g[j] = h;
  }
  dst[step - 1] = par;
  if (g) g[step - 1] = par;
}

// Copies one step's records into the arena: k and v rows move as 16-byte
// chunks from beam-major [R][W][H][d] to slab-major
// [R][tmax][H][wmax][d] (destination order, so writes are contiguous);
// (alpha, beta) are interleaved into one 8-byte pair per (slot, value head).
struct AppendArgs {
  const uint4* k;
  const uint4* v;
  const float* alpha;
  const float* beta;
  uint4* ak;
  uint4* av;
  float2* aab;
  int R, HK, HV, width, wmax, tmax, step;
  int cpr_k, cpr_v;       // 16-byte chunks per k / v row
  long nk, nv, nab;       // work items of each part
};

__global__ void append_kernel(AppendArgs a) {
  const long i = long(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < a.nk) {
    // destination order (r, h, b, c)
    const int c = int(i % a.cpr_k);
    long rest = i / a.cpr_k;
    const int b = int(rest % a.width);
    rest /= a.width;
    const int h = int(rest % a.HK);
    const int r = int(rest / a.HK);
    const long src = ((long(r) * a.width + b) * a.HK + h) * a.cpr_k + c;
    const long dst = (((long(r) * a.tmax + a.step) * a.HK + h) * a.wmax + b) * a.cpr_k + c;
    a.ak[dst] = a.k[src];
    return;
  }
  long j = i - a.nk;
  if (j < a.nv) {
    const int c = int(j % a.cpr_v);
    long rest = j / a.cpr_v;
    const int b = int(rest % a.width);
    rest /= a.width;
    const int h = int(rest % a.HV);
    const int r = int(rest / a.HV);
    const long src = ((long(r) * a.width + b) * a.HV + h) * a.cpr_v + c;
    const long dst = (((long(r) * a.tmax + a.step) * a.HV + h) * a.wmax + b) * a.cpr_v + c;
    a.av[dst] = a.v[src];
    return;
  }
  j -= a.nv;
  if (j < a.nab) {
    const int b = int(j % a.width);
    long rest = j / a.width;
    const int h = int(rest % a.HV);
    const int r = int(rest / a.HV);
    const long src = (long(r) * a.width + b) * a.HV + h;
    const long dst = ((long(r) * a.tmax + a.step) * a.HV + h) * a.wmax + b;
    a.aab[dst] = make_float2(a.alpha[src], a.beta[src]);
  }
}

unsigned blocks_for(long n, int threads) { return unsigned((n + threads - 1) / threads); }

}  // namespace

hipError_t launch_clear_status(int* status, hipStream_t st) {
  clear_status_kernel<<<1, 64, 0, st>>>(status);
  return hipGetLastError();
}

hipError_t launch_resolve(const Shape& s, int step, int width, int prev_width,
                          const int* parents, const int* anc_prev, int* anc_cur,
                          int* gather_out, int* status, hipStream_t st) {
  const long n = long(s.R) * width;
  resolve_kernel<<<blocks_for(n, 256), 256, 0, st>>>(parents, anc_prev, anc_cur, gather_out,
                                                     status, s.R, width, prev_width, s.wmax,
                                                     s.tmax, step);
  return hipGetLastError();
}

hipError_t launch_append(const Shape& s, int step, int width, const void* k, const void* v,
                         const float* alpha, const float* beta, const Arena& ar,
                         hipStream_t st) {
  AppendArgs a;
  a.k = static_cast<const uint4*>(k);
  a.v = static_cast<const uint4*>(v);
  a.alpha = alpha;
  a.beta = beta;
  a.ak = static_cast<uint4*>(ar.k);
  a.av = static_cast<uint4*>(ar.v);
  a.aab = ar.ab;
  a.R = s.R;
  a.HK = s.HK;
  a.HV = s.HV;
  a.width = width;
  a.wmax = s.wmax;
  a.tmax = s.tmax;
  a.step = step;
  a.cpr_k = s.dk * s.io_bytes() / 16;
  a.cpr_v = s.dv * s.io_bytes() / 16;
  a.nk = long(s.R) * width * s.HK * a.cpr_k;
  a.nv = long(s.R) * width * s.HV * a.cpr_v;
  a.nab = long(s.R) * width * s.HV;
  append_kernel<<<blocks_for(a.nk + a.nv + a.nab, 256), 256, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace onela
