// Fused large-beam GDN decode step for gfx950 (CDNA4).
//
// For every request r, value head hv and live beam b, with the chain of
// records (k_j, v_j, alpha_j, beta_j) at slots h_t(b, 0..t-1) of steps
// 0..t-1 plus the beam's own step-t record (Sec. 3.3, Eq. 5), the kernel
// computes the Eq. 1 read-out o = S_{t,b} q without forming S_{t,b}.
//
// Algebra.  Eq. 1 is S_j = S_{j-1} A_j + beta_j v_j k_j^T with
// A_j = alpha_j (I - beta_j k_j k_j^T).  Folding the query newest to oldest,
//     p <- q;  for j = t..0:  c = k_j . p;  g_j = beta_j c;
//                             o += g_j v_j;  p <- alpha_j (p - g_j k_j)
//     o += S_ctx p,
// gives S_{t,b} q exactly (in exact arithmetic).  The only d_v x d_k work is
// the final S_ctx p, which is a dense GEMM over all beams of a head:
// O_h = S_ctx[h] . [p_1 .. p_W].  That contraction runs on MFMA; the fold and
// the v-terms are vector work with 16-byte loads.
//
// Precision.  S_ctx is split once (at init) into bf16 hi + lo, p is split the
// same way in registers, and O = S_hi P_hi + S_hi P_lo + S_lo P_hi is
// accumulated in fp32 by v_mfma_f32_16x16x32_bf16 (about 16 significant bits
// per product; the dropped S_lo P_lo term is ~2^-17 relative).
//
// Work decomposition.  One workgroup = (request, value head, 16*NBLK beams),
// DV/32 waves.  Phase 1 (fold): LPB lanes per beam, each owning EPL
// consecutive key elements; dot products are reduced across those lanes.
// The folded queries are written, split into hi/lo, to LDS directly in MFMA
// B-fragment order; the fold scalars g_j go to LDS too.  Phase 2 (contract):
// wave w multiplies its 32 state rows (A fragments streamed from the
// fragment-ordered split state, issued before the fold so they overlap it)
// by the beams' B fragments.  Phase 3 (epilogue): each lane holds 8
// consecutive output rows of one beam, adds sum_j g_j v_j[rows] (v prefetched
// at kernel start) and stores 32 contiguous bytes.
//
// Block order is XCD-aware: workgroups are dispatched round-robin over the 8
// XCDs, so block id i runs on XCD i % 8; all beam tiles of a (request, head)
// are mapped to one XCD so that head's shared state and records stay in that
// XCD's L2.
#include "internal.h"

namespace onela {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct DecodeParams {
  const void* q;
  float* o;
  const uint4* s_frag;
  const void* ak;
  const void* av;
  const float2* ab;
  const int* anc;
  int R, HK, HV, W, wmax, tmax;
  int ntiles;   // beam tiles per (request, value head)
  int xcd_map;  // 1: XCD-aware block order (units % 8 == 0)
};

// 8 consecutive io elements, raw.
template <bool BF16>
struct Raw8;
template <>
struct Raw8<true> {
  uint4 u;
  __device__ void load(const void* base, long elem) {
    u = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + elem);
  }
  __device__ void to_float(float* x) const {
    x[0] = __uint_as_float(u.x << 16);
    x[1] = __uint_as_float(u.x & 0xffff0000u);
    x[2] = __uint_as_float(u.y << 16);
    x[3] = __uint_as_float(u.y & 0xffff0000u);
    x[4] = __uint_as_float(u.z << 16);
    x[5] = __uint_as_float(u.z & 0xffff0000u);
    x[6] = __uint_as_float(u.w << 16);
    x[7] = __uint_as_float(u.w & 0xffff0000u);
  }
};
template <>
struct Raw8<false> {
  float4 a, b;
  __device__ void load(const void* base, long elem) {
    const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(base) + elem);
    a = p[0];
    b = p[1];
  }
  __device__ void to_float(float* x) const {
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  }
};

__device__ inline unsigned pack_bf16x2(float a, float b) {
  return unsigned(__builtin_bit_cast(unsigned short, static_cast<__bf16>(a))) |
         (unsigned(__builtin_bit_cast(unsigned short, static_cast<__bf16>(b))) << 16);
}

__device__ inline float bf16_lo_to_float(unsigned u) { return __uint_as_float(u << 16); }
__device__ inline float bf16_hi_to_float(unsigned u) { return __uint_as_float(u & 0xffff0000u); }

// Split 8 floats into bf16 hi and lo vectors: hi = bf16(x), lo = bf16(x - hi).
__device__ inline void split8(const float* x, uint4& hi, uint4& lo) {
  unsigned h[4], l[4];
  for (int i = 0; i < 4; ++i) {
    h[i] = pack_bf16x2(x[2 * i], x[2 * i + 1]);
    l[i] = pack_bf16x2(x[2 * i] - bf16_lo_to_float(h[i]),
                       x[2 * i + 1] - bf16_hi_to_float(h[i]));
  }
  hi = make_uint4(h[0], h[1], h[2], h[3]);
  lo = make_uint4(l[0], l[1], l[2], l[3]);
}

__device__ inline f32x4 mfma_bf16(const uint4& a, const uint4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

template <int DK, int DV, int NBLK, int CHAIN, bool BF16>
__global__ __launch_bounds__(DV * 2) void decode_kernel(DecodeParams p) {
  constexpr int NW = DV / 32;        // waves per workgroup
  constexpr int NT = NW * 64;        // threads per workgroup
  constexpr int BEAMS = 16 * NBLK;   // beams per workgroup
  constexpr int LPB = NT / BEAMS;    // fold lanes per beam
  constexpr int EPL = DK / LPB;      // key elements per fold lane
  constexpr int C8 = EPL / 8;        // 8-element chunks per fold lane
  constexpr int KS = DK / 32;        // MFMA k-steps
  static_assert(EPL % 8 == 0 && EPL >= 8, "fold lanes must own 8-element chunks");
  static_assert(LPB <= 64 && (LPB & (LPB - 1)) == 0, "fold lane group within a wave");

  __shared__ uint4 p_lds[2][NBLK][KS][4][16];  // folded queries, B-fragment order
  __shared__ float g_lds[BEAMS][CHAIN];        // fold scalars g_j

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;

  int unit, tile;
  if (p.xcd_map) {
    const int x = blockIdx.x & 7, slot = blockIdx.x >> 3;
    unit = x + 8 * (slot / p.ntiles);
    tile = slot % p.ntiles;
  } else {
    unit = blockIdx.x / p.ntiles;
    tile = blockIdx.x % p.ntiles;
  }
  const int r = unit / p.HV;
  const int hv = unit - r * p.HV;
  const int hk = hv / (p.HV / p.HK);
  const int b0 = tile * BEAMS;
  const int W = p.W;

  // ---- A fragments of this wave's 32 state rows (independent of the beams)
  uint4 A[KS][2][2];
  {
    const uint4* sf = p.s_frag + (long(unit) * NW + w) * (KS * 4 * 64) + lane;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int hl = 0; hl < 2; ++hl) A[ks][mb][hl] = sf[((ks * 2 + mb) * 2 + hl) * 64];
  }

  // ---- fold-phase lane mapping and chain slots
  const int fb = tid / LPB;
  const int li = tid - fb * LPB;
  const int fbeam = b0 + fb;
  const int fbc = fbeam < W ? fbeam : 0;
  int fslot[CHAIN];
  bool fok[CHAIN];
  {
    const int* arow = p.anc + (long(r) * p.wmax + fbc) * p.tmax;
#pragma unroll
    for (int j = 0; j < CHAIN - 1; ++j) {
      const int s = arow[j];
      fok[j] = unsigned(s) < unsigned(p.wmax);
      fslot[j] = fok[j] ? s : 0;
    }
    fslot[CHAIN - 1] = fbc;
    fok[CHAIN - 1] = true;
  }

  // ---- epilogue lane mapping and chain slots (one beam per lane and block)
  const int g4 = lane >> 4;  // 8-row group of this lane within the wave's rows
  int sslot[NBLK][CHAIN];
#pragma unroll
  for (int nb = 0; nb < NBLK; ++nb) {
    const int sb = b0 + nb * 16 + (lane & 15);
    const int sbc = sb < W ? sb : 0;
    const int* arow = p.anc + (long(r) * p.wmax + sbc) * p.tmax;
#pragma unroll
    for (int j = 0; j < CHAIN - 1; ++j) {
      const int s = arow[j];
      sslot[nb][j] = unsigned(s) < unsigned(p.wmax) ? s : 0;
    }
    sslot[nb][CHAIN - 1] = sbc;
  }

  // ---- issue every beam-side load up front
  Raw8<BF16> qr[C8];
  Raw8<BF16> kr[CHAIN][C8];
  float2 abr[CHAIN];
  Raw8<BF16> vr[NBLK][CHAIN];
  {
    const long qbase = ((long(r) * W + fbc) * p.HK + hk) * DK + li * EPL;
#pragma unroll
    for (int c = 0; c < C8; ++c) qr[c].load(p.q, qbase + 8 * c);
#pragma unroll
    for (int j = 0; j < CHAIN; ++j) {
      const long slab = long(r) * p.tmax + j;
      const long kbase = ((slab * p.HK + hk) * p.wmax + fslot[j]) * DK + li * EPL;
#pragma unroll
      for (int c = 0; c < C8; ++c) kr[j][c].load(p.ak, kbase + 8 * c);
      abr[j] = p.ab[(slab * p.HV + hv) * p.wmax + fslot[j]];
    }
#pragma unroll
    for (int nb = 0; nb < NBLK; ++nb)
#pragma unroll
      for (int j = 0; j < CHAIN; ++j) {
        const long slab = long(r) * p.tmax + j;
        vr[nb][j].load(p.av, ((slab * p.HV + hv) * p.wmax + sslot[nb][j]) * DV + 32 * w + 8 * g4);
      }
  }

  // ---- phase 1: fold the query newest -> oldest
  float pv[EPL];
#pragma unroll
  for (int c = 0; c < C8; ++c) qr[c].to_float(pv + 8 * c);
#pragma unroll
  for (int j = CHAIN - 1; j >= 0; --j) {
    float kf[EPL];
#pragma unroll
    for (int c = 0; c < C8; ++c) kr[j][c].to_float(kf + 8 * c);
    float c0 = 0.f, c1 = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; e += 2) {
      c0 = fmaf(kf[e], pv[e], c0);
      c1 = fmaf(kf[e + 1], pv[e + 1], c1);
    }
    float cdot = c0 + c1;
#pragma unroll
    for (int m = 1; m < LPB; m <<= 1) cdot += __shfl_xor(cdot, m);
    const float alpha = fok[j] ? abr[j].x : 1.f;
    const float beta = fok[j] ? abr[j].y : 0.f;
    const float gj = beta * cdot;
    if (li == 0) g_lds[fb][j] = gj;
#pragma unroll
    for (int e = 0; e < EPL; ++e) pv[e] = alpha * fmaf(-gj, kf[e], pv[e]);
  }
#pragma unroll
  for (int c = 0; c < C8; ++c) {
    const int k0 = li * EPL + 8 * c;
    uint4 hi, lo;
    split8(pv + 8 * c, hi, lo);
    p_lds[0][fb >> 4][k0 >> 5][(k0 >> 3) & 3][fb & 15] = hi;
    p_lds[1][fb >> 4][k0 >> 5][(k0 >> 3) & 3][fb & 15] = lo;
  }
  __syncthreads();

  // ---- phase 2: O = S_ctx . P on MFMA (three bf16 products per block)
  f32x4 acc[NBLK][2];
#pragma unroll
  for (int nb = 0; nb < NBLK; ++nb) {
    acc[nb][0] = f32x4{0.f, 0.f, 0.f, 0.f};
    acc[nb][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const uint4 bh = p_lds[0][nb][ks][g4][lane & 15];
      const uint4 bl = p_lds[1][nb][ks][g4][lane & 15];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        acc[nb][mb] = mfma_bf16(A[ks][mb][1], bh, acc[nb][mb]);
        acc[nb][mb] = mfma_bf16(A[ks][mb][0], bl, acc[nb][mb]);
        acc[nb][mb] = mfma_bf16(A[ks][mb][0], bh, acc[nb][mb]);
      }
    }
  }

  // ---- phase 3: add the v-terms and store 8 consecutive rows per lane
#pragma unroll
  for (int nb = 0; nb < NBLK; ++nb) {
    const int bl = nb * 16 + (lane & 15);
    const int sb = b0 + bl;
    float ov[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) ov[e] = acc[nb][e >> 2][e & 3];
#pragma unroll
    for (int j = 0; j < CHAIN; ++j) {
      const float gj = g_lds[bl][j];
      float vf[8];
      vr[nb][j].to_float(vf);
#pragma unroll
      for (int e = 0; e < 8; ++e) ov[e] = fmaf(gj, vf[e], ov[e]);
    }
    if (sb < W) {
      float4* dst = reinterpret_cast<float4*>(p.o + ((long(r) * W + sb) * p.HV + hv) * DV +
                                              32 * w + 8 * g4);
      dst[0] = make_float4(ov[0], ov[1], ov[2], ov[3]);
      dst[1] = make_float4(ov[4], ov[5], ov[6], ov[7]);
    }
  }
}

template <int D, int NBLK, bool BF16>
hipError_t launch_chain(int chain, const DecodeParams& prm, unsigned blocks, hipStream_t st) {
  constexpr int threads = D * 2;
  switch (chain) {
#define ONELA_CHAIN_CASE(C)                                                          \
  case C:                                                                           \
    decode_kernel<D, D, NBLK, C, BF16><<<blocks, threads, 0, st>>>(prm);            \
    break;
    ONELA_CHAIN_CASE(1)
    ONELA_CHAIN_CASE(2)
    ONELA_CHAIN_CASE(3)
    ONELA_CHAIN_CASE(4)
    ONELA_CHAIN_CASE(5)
    ONELA_CHAIN_CASE(6)
    ONELA_CHAIN_CASE(7)
    ONELA_CHAIN_CASE(8)
#undef ONELA_CHAIN_CASE
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

bool decode_supported(const Shape& s) {
  return s.dk == s.dv && (s.dk == 32 || s.dk == 64 || s.dk == 128);
}

hipError_t launch_decode(const Shape& s, int step, int width, const void* q, float* o,
                         const Arena& a, hipStream_t st) {
  constexpr int NBLK = 1;
  DecodeParams prm;
  prm.q = q;
  prm.o = o;
  prm.s_frag = reinterpret_cast<const uint4*>(a.s_frag);
  prm.ak = a.k;
  prm.av = a.v;
  prm.ab = a.ab;
  prm.anc = a.anc[step & 1];
  prm.R = s.R;
  prm.HK = s.HK;
  prm.HV = s.HV;
  prm.W = width;
  prm.wmax = s.wmax;
  prm.tmax = s.tmax;
  prm.ntiles = (width + 16 * NBLK - 1) / (16 * NBLK);
  const int units = s.R * s.HV;
  prm.xcd_map = (units % 8 == 0) ? 1 : 0;
  const unsigned blocks = unsigned(units) * unsigned(prm.ntiles);
  const int chain = step + 1;
  if (s.dk == 128)
    return s.bf16 ? launch_chain<128, NBLK, true>(chain, prm, blocks, st)
                  : launch_chain<128, NBLK, false>(chain, prm, blocks, st);
  if (s.dk == 64)
    return s.bf16 ? launch_chain<64, NBLK, true>(chain, prm, blocks, st)
                  : launch_chain<64, NBLK, false>(chain, prm, blocks, st);
  if (s.dk == 32)
    return s.bf16 ? launch_chain<32, NBLK, true>(chain, prm, blocks, st)
                  : launch_chain<32, NBLK, false>(chain, prm, blocks, st);
  return hipErrorInvalidValue;
}

}  // namespace onela
