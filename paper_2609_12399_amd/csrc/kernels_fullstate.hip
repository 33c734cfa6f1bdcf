// Materialised-state GDN kernels (gfx950): the prompt prefill that produces
// S_ctx, and the per-beam "FullState" decode baseline.  Both keep the fp32
// state rows of one (request, value head[, beam]) in the registers of
// 256-thread workgroups and apply Eq. 1 (Sec. 2.2) literally:
//     u = S k;  S <- alpha S + beta (v - alpha u) k^T;  o = S q.
// Thread layout: LPR = d_k/4 lanes per state row, each owning 4 consecutive
// columns (one 16-byte vector); a pass covers 256/LPR rows.  Rows of Eq. 1
// are independent (u_i = S_i k, S_i <- alpha S_i + w_i k^T), so wide states
// are split into row slices of at most 16 passes, one workgroup each.  Row
// sums are reduced across the LPR lanes.
#include <type_traits>

#include "internal.h"

namespace onela {
namespace {

constexpr int kThreads = 256;

template <bool BF16>
__device__ inline float4 load4(const void* base, long elem) {
  if constexpr (BF16) {
    const uint2 u = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(base) + elem);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                       __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
  } else {
    return *reinterpret_cast<const float4*>(static_cast<const float*>(base) + elem);
  }
}

template <bool BF16>
__device__ inline float load1(const void* base, long elem) {
  if constexpr (BF16) {
    return __uint_as_float(unsigned(static_cast<const uint16_t*>(base)[elem]) << 16);
  } else {
    return static_cast<const float*>(base)[elem];
  }
}

template <int LPR>
__device__ inline float row_sum(float x) {
#pragma unroll
  for (int m = 1; m < LPR; m <<= 1) x += __shfl_xor(x, m);
  return x;
}

__device__ inline float dot4(const float4& a, const float4& b) {
  return fmaf(a.x, b.x, fmaf(a.y, b.y, fmaf(a.z, b.z, a.w * b.w)));
}

// One Eq. 1 transition on a register-resident state.  vrow[pass] is v at the
// thread's row of that pass.
template <int LPR, int NP>
__device__ inline void transition(float4 (&S)[NP], const float4& kc, const float (&vrow)[NP],
                                  float alpha, float beta) {
#pragma unroll
  for (int ps = 0; ps < NP; ++ps) {
    const float u = row_sum<LPR>(dot4(S[ps], kc));
    const float wv = beta * (vrow[ps] - alpha * u);
    S[ps].x = fmaf(alpha, S[ps].x, wv * kc.x);
    S[ps].y = fmaf(alpha, S[ps].y, wv * kc.y);
    S[ps].z = fmaf(alpha, S[ps].z, wv * kc.z);
    S[ps].w = fmaf(alpha, S[ps].w, wv * kc.w);
  }
}

// Rows per workgroup for a d_k x d_v state: at most 16 passes.
template <int DK, int DV>
constexpr int slice_rows() {
  constexpr int rpp = kThreads / (DK / 4);
  return DV < 16 * rpp ? DV : 16 * rpp;
}

// Prefill: one workgroup per (request, value head, row slice), tokens in
// order.
template <int DK, int DV, bool BF16>
__global__ __launch_bounds__(kThreads) void prefill_kernel(const void* __restrict__ k,
                                                           const void* __restrict__ v,
                                                           const float* __restrict__ alpha,
                                                           const float* __restrict__ beta,
                                                           float* __restrict__ s_out, int HK,
                                                           int HV, int P) {
  constexpr int LPR = DK / 4, RPP = kThreads / LPR, ROWS = slice_rows<DK, DV>();
  constexpr int NP = ROWS / RPP, NSL = DV / ROWS;
  static_assert(NP >= 1 && ROWS % RPP == 0 && DV % ROWS == 0, "state must tile the workgroup");
  const int unit = blockIdx.x / NSL, sl = blockIdx.x % NSL;
  const int r = unit / HV, hv = unit - r * HV, hk = hv / (HV / HK);
  const int rr = threadIdx.x / LPR, cc = threadIdx.x % LPR;
  const int rbase = sl * ROWS;
  float4 S[NP];
#pragma unroll
  for (int ps = 0; ps < NP; ++ps) S[ps] = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int t = 0; t < P; ++t) {
    const long tok = long(r) * P + t;
    const float4 kc = load4<BF16>(k, (tok * HK + hk) * DK + 4 * cc);
    float vrow[NP];
#pragma unroll
    for (int ps = 0; ps < NP; ++ps)
      vrow[ps] = load1<BF16>(v, (tok * HV + hv) * DV + rbase + ps * RPP + rr);
    const float a = alpha[tok * HV + hv], b = beta[tok * HV + hv];
    transition<LPR, NP>(S, kc, vrow, a, b);
  }
#pragma unroll
  for (int ps = 0; ps < NP; ++ps)
    reinterpret_cast<float4*>(s_out + (long(unit) * DV + rbase + ps * RPP + rr) * DK)[cc] = S[ps];
}

// FullState decode baseline: one workgroup per (request, beam, value head,
// row slice).
template <int DK, int DV, bool BF16>
__global__ __launch_bounds__(kThreads) void fullstate_kernel(
    const int* __restrict__ parents, const float* __restrict__ s0, const void* __restrict__ q,
    const void* __restrict__ k, const void* __restrict__ v, const float* __restrict__ alpha,
    const float* __restrict__ beta, float* __restrict__ o, const float* __restrict__ st_in,
    float* __restrict__ st_out, int* __restrict__ status, int HK, int HV, int width,
    int prev_width, int wmax, int step) {
  constexpr int LPR = DK / 4, RPP = kThreads / LPR, ROWS = slice_rows<DK, DV>();
  constexpr int NP = ROWS / RPP, NSL = DV / ROWS;
  const int sl = blockIdx.x % NSL;
  const int hv = (blockIdx.x / NSL) % HV;
  const int rb = blockIdx.x / NSL / HV;  // r * width + b
  const int r = rb / width, b = rb - r * width;
  const int hk = hv / (HV / HK);
  const int rr = threadIdx.x / LPR, cc = threadIdx.x % LPR;
  const int rbase = sl * ROWS;
  const float* src;
  if (step == 0) {
    src = s0 + (long(r) * HV + hv) * DV * DK;
  } else {
    int par = parents[rb];
    if (par < 0 || par >= prev_width) {
      if (status && threadIdx.x == 0) atomicOr(status, kStatusParent);
      par = 0;
    }
    src = st_in + ((long(r) * wmax + par) * HV + hv) * DV * DK;
  }
  float4 S[NP];
#pragma unroll
  for (int ps = 0; ps < NP; ++ps)
    S[ps] = reinterpret_cast<const float4*>(src + long(rbase + ps * RPP + rr) * DK)[cc];
  const long tok = long(r) * width + b;
  const float4 kc = load4<BF16>(k, (tok * HK + hk) * DK + 4 * cc);
  const float4 qc = load4<BF16>(q, (tok * HK + hk) * DK + 4 * cc);
  float vrow[NP];
#pragma unroll
  for (int ps = 0; ps < NP; ++ps)
    vrow[ps] = load1<BF16>(v, (tok * HV + hv) * DV + rbase + ps * RPP + rr);
  transition<LPR, NP>(S, kc, vrow, alpha[tok * HV + hv], beta[tok * HV + hv]);
  float* dst = st_out + ((long(r) * wmax + b) * HV + hv) * DV * DK;
#pragma unroll
  for (int ps = 0; ps < NP; ++ps) {
    reinterpret_cast<float4*>(dst + long(rbase + ps * RPP + rr) * DK)[cc] = S[ps];
    const float oi = row_sum<LPR>(dot4(S[ps], qc));
    if (cc == 0) o[(tok * HV + hv) * DV + rbase + ps * RPP + rr] = oi;
  }
}

template <int DK, int DV, bool BF16>
void launch_prefill_t(const Shape& s, int P, const void* k, const void* v, const float* a,
                      const float* b, float* out, hipStream_t st) {
  const unsigned blocks = unsigned(s.R * s.HV) * unsigned(DV / slice_rows<DK, DV>());
  prefill_kernel<DK, DV, BF16><<<blocks, kThreads, 0, st>>>(k, v, a, b, out, s.HK, s.HV, P);
}

template <int DK, int DV, bool BF16>
void launch_fullstate_t(const Shape& s, int step, int width, int prev_width, const int* par,
                        const float* s0, const void* q, const void* k, const void* v,
                        const float* a, const float* b, float* o, const float* in, float* out,
                        int* status, hipStream_t st) {
  const unsigned blocks =
      unsigned(s.R) * unsigned(width) * unsigned(s.HV) * unsigned(DV / slice_rows<DK, DV>());
  fullstate_kernel<DK, DV, BF16><<<blocks, kThreads, 0, st>>>(
      par, s0, q, k, v, a, b, o, in, out, status, s.HK, s.HV, width, prev_width, s.wmax, step);
}

// The (d_k, d_v, io) combinations the library accepts (see decode_supported).
template <typename F>
hipError_t dispatch_shape(const Shape& s, F&& f) {
#define ONELA_FS_SHAPE(DK, DV)                                                 \
  if (s.dk == DK && s.dv == DV) {                                             \
    if (s.bf16) f(std::integral_constant<int, DK>(), std::integral_constant<int, DV>(), \
                  std::true_type());                                          \
    else f(std::integral_constant<int, DK>(), std::integral_constant<int, DV>(),        \
           std::false_type());                                                \
    return hipGetLastError();                                                 \
  }
  ONELA_FS_SHAPE(32, 32)
  ONELA_FS_SHAPE(64, 64)
  ONELA_FS_SHAPE(128, 128)
  ONELA_FS_SHAPE(128, 256)
  ONELA_FS_SHAPE(128, 512)
  ONELA_FS_SHAPE(256, 256)
  ONELA_FS_SHAPE(256, 512)
#undef ONELA_FS_SHAPE
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_prefill(const Shape& s, int prompt_len, const void* k, const void* v,
                          const float* alpha, const float* beta, float* s0_out,
                          hipStream_t st) {
  return dispatch_shape(s, [&](auto DK, auto DV, auto BF16) {
    launch_prefill_t<decltype(DK)::value, decltype(DV)::value, decltype(BF16)::value>(
        s, prompt_len, k, v, alpha, beta, s0_out, st);
  });
}

hipError_t launch_fullstate(const Shape& s, int step, int width, int prev_width,
                            const int* parents, const float* s0, const void* q, const void* k,
                            const void* v, const float* alpha, const float* beta, float* o,
                            const float* states_in, float* states_out, int* status,
                            hipStream_t st) {
  return dispatch_shape(s, [&](auto DK, auto DV, auto BF16) {
    launch_fullstate_t<decltype(DK)::value, decltype(DV)::value, decltype(BF16)::value>(
        s, step, width, prev_width, parents, s0, q, k, v, alpha, beta, o, states_in,
        states_out, status, st);
  });
}

}  // namespace onela
