// Large-beam GDN decode step with the paper's transition records (gfx950).
//
// Records are the GDN transition records of Sec. 3.2, r_j = (alpha_j, delta_j,
// k_j) with delta_j = beta_j (v_j - alpha_j S_{j-1} k_j) (Eq. 2), stored once
// per (step, slot) and never moved.  A decode step replays the beam's
// ancestral records onto the two projections it needs (Eq. 3):
//     u_q = S_ctx q_t,  u_k = S_ctx k_t;
//     for j = 0..t-1:  u_q <- alpha_j u_q + delta_j (k_j . q_t)
//                      u_k <- alpha_j u_k + delta_j (k_j . k_t)
// and evaluates the step (Eq. 4):
//     delta_t = beta_t (v_t - alpha_t u_k),  o_t = alpha_t u_q + delta_t (k_t . q_t),
// appending r_t = (alpha_t, delta_t, k_t).  Unrolled, u = (prod_j alpha_j) S x
// + sum_j w_j delta_j with w_j = (k_j . x) prod_{i>j} alpha_i, so every record
// contributes independently: one dot product per (record, projection) and one
// weighted d_v-vector per record.
//
// Layout of the work is the one of the input-record decode kernel (one
// workgroup = request, value head, row slice, 32 beams; d_k/16 waves of 16*MB
// state rows; XCD-aware block order; shared state split into bf16 hi/lo,
// stored split by step 0).  The difference is the order of dependencies:
// the contraction S_ctx [q_t | k_t] needs no record, so after one barrier
// (the B fragments of q_t and k_t staged in LDS) the MFMAs run while the
// ancestral records are still arriving; the record dots follow.  As in the
// input-record kernel, every load is made by the fold lanes of the beam as
// whole lines: each lane forms sum_j w_j delta_j for both projections over its
// value rows and stages them, with v_t, in LDS; a second barrier publishes
// them, and the epilogue applies Eq. 4 in the MFMA output layout.
//
// delta is stored in fp16 for bf16 inputs (fp32 for fp32 inputs): the paper's
// record is a 32-bit decay with 16-bit delta and key vectors; bf16 would cost
// ~8x more error.  fp16 alone would bound the magnitudes the inputs may have
// (values above 65504 overflow, values below 2^-14 lose bits), so each row
// slice of delta_t is stored divided by 2^e, with e chosen from the slice's
// largest magnitude (which then lies in [2^14, 2^15)); e is kept as an int8
// per slice, four to a 32-bit word per row.  MODE: DECODE reads the step-t record from the arena (after
// onela_append_records); FUSED reads it from the caller and performs the
// ancestry update and the append in the same launch.
#include "device_common.h"
#include "internal.h"

namespace onela {
namespace {

struct ReplayParams {
  const void* q;
  float* o;
  const int* parents;  // FUSED
  const void* k_in;    // FUSED: the step's inputs
  const void* v_in;
  const float* alpha_in;
  const float* beta_in;
  int* gather_out;
  int* status;
  const float* s0;
  uint4* s_frag;
  void* ak;    // arena keys [R][tmax][HK][wmax][dk] io dtype
  void* av;    // arena step inputs v (DECODE mode reads step t from here)
  float2* ab;  // arena (alpha, beta)
  void* ad;    // arena delta [R][tmax][HV][wmax][dv], fp16 (bf16 io) or fp32
  unsigned* adsc;  // arena delta scale exponents [R][tmax][HV][wmax], int8 per slice
  const int* anc_rd;
  int* anc_wr;
  int R, HK, HV, G, W, W_prev, wmax, tmax;
  int ntiles;
  int xcd_map;
};

// delta rows: fp16 words for bf16 inputs, fp32 otherwise (same byte sizes as
// the input rows, so RawV moves them).
template <bool F16>
__device__ inline void delta_to_float(const unsigned* w, float* x, int n) {
  for (int i = 0; i < (F16 ? n / 2 : n); ++i) {
    if constexpr (F16) {
      x[2 * i] = float(__builtin_bit_cast(_Float16, static_cast<unsigned short>(w[i] & 0xffffu)));
      x[2 * i + 1] = float(__builtin_bit_cast(_Float16, static_cast<unsigned short>(w[i] >> 16)));
    } else {
      x[i] = __uint_as_float(w[i]);
    }
  }
}

template <bool F16>
__device__ inline void float_to_delta(const float* x, unsigned* w, int n) {
  for (int i = 0; i < (F16 ? n / 2 : n); ++i) {
    if constexpr (F16) {
      const unsigned lo = __builtin_bit_cast(unsigned short, static_cast<_Float16>(x[2 * i]));
      const unsigned hi = __builtin_bit_cast(unsigned short, static_cast<_Float16>(x[2 * i + 1]));
      w[i] = lo | (hi << 16);
    } else {
      w[i] = __float_as_uint(x[i]);
    }
  }
}

template <int DK, int DV, int DVW, int NBLK, int CHAIN, bool BF16, bool FUSED>
__global__ __launch_bounds__(4 * DK) void replay_kernel(ReplayParams p) {
  constexpr int MB = DVW / DK;
  constexpr int NS = DV / DVW;
  constexpr int NW = DVW / (16 * MB);
  constexpr int RPL = 4 * MB;
  constexpr int NT = NW * 64;
  constexpr int BEAMS = 16 * NBLK;
  constexpr int LPB = NT / BEAMS;    // fold lanes per beam
  constexpr int EPL = DK / LPB;      // key elements per fold lane
  constexpr int C8 = EPL / 8;
  constexpr int VPL = DVW / LPB;     // value rows per fold lane
  constexpr int VS = DVW + 4;        // padded LDS row per beam
  constexpr int KS = DK / 32;
  constexpr int NA = CHAIN - 1;
  constexpr int NAX = NA > 0 ? NA : 1;
  constexpr unsigned IOB = BF16 ? 2 : 4;
  constexpr int HL = BF16 ? 1 : 2;   // bf16 inputs are exact in bf16: no low half
  static_assert(MB * DK == DVW && NS * DVW == DV && EPL % 8 == 0, "tiling");
  static_assert(LPB <= 64 && (LPB & (LPB - 1)) == 0, "fold lane group within a wave");
  static_assert(VPL == 8 || VPL == 16, "fold lanes own 8 or 16 value rows");

  __shared__ uint4 b_lds[2][HL][NBLK][KS][4][16];  // [q | k_t][hi | lo] B fragments
  __shared__ float sc_lds[BEAMS][4];               // decay, alpha_t, beta_t, k_t.q
  // per beam and row of this slice: sum_j w_q,j delta_j, sum_j w_k,j delta_j, v_t
  __shared__ float rq_lds[BEAMS][VS], rk_lds[BEAMS][VS], vt_lds[BEAMS][VS];
  // FUSED, t >= 2: columns 0..t-2 of the request's h_{t-1}, all previous beams
  constexpr bool kTab = FUSED && NA >= 2;
  constexpr int NL = NT < 256 ? NT : 256;  // table-loading threads (at most 4 waves)
  constexpr int NTV = kAncTable / NL;      // table entries per loading lane
  __shared__ int anc_lds[kTab ? kAncTable : 1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  // the arguments the first loads depend on, in scalar registers together
  // (one round of argument loads; see the input-record kernel)
  if constexpr (FUSED)
    asm volatile("" ::"s"(p.ntiles), "s"(p.xcd_map), "s"(p.HK), "s"(p.HV), "s"(p.G), "s"(p.W),
                 "s"(p.wmax), "s"(p.tmax), "s"(p.anc_rd), "s"(p.q), "s"(p.W_prev), "s"(p.parents),
                 "s"(p.k_in), "s"(p.v_in), "s"(p.alpha_in), "s"(p.beta_in), "s"(p.ak), "s"(p.ad),
                 "s"(p.ab));
  else
    asm volatile("" ::"s"(p.ntiles), "s"(p.xcd_map), "s"(p.HK), "s"(p.HV), "s"(p.G), "s"(p.W),
                 "s"(p.wmax), "s"(p.tmax), "s"(p.anc_rd), "s"(p.q), "s"(p.ak), "s"(p.av),
                 "s"(p.ad), "s"(p.ab));
  if constexpr (NA == 0) {
    if (blockIdx.x == 0 && tid == 0) p.status[0] = 0;
  }

  int unit, st;
  const int nst = NS * p.ntiles;
  if (p.xcd_map) {
    const int x = blockIdx.x & 7, slot = blockIdx.x >> 3;
    unit = x + 8 * (slot / nst);
    st = slot % nst;
  } else {
    unit = blockIdx.x / nst;
    st = blockIdx.x % nst;
  }
  const int slice = st / p.ntiles;
  const int tile = st - slice * p.ntiles;
  const int r = unit / p.HV;
  const int hv = unit - r * p.HV;
  const int hk = hv / p.G;
  const int b0 = tile * BEAMS;
  const int W = p.W;
  const int wmax = p.wmax, tmax = p.tmax;

  const int fb = tid / LPB;
  const int li = tid - fb * LPB;
  const int fbeam = b0 + fb;
  const bool fvalid = fbeam < W;
  const int fbc = fvalid ? fbeam : 0;
  const unsigned voff = (unsigned(DVW) * slice + unsigned(li) * VPL) * IOB;
  const int g4 = lane >> 4;
  const unsigned rloc = 16 * MB * w + RPL * g4;  // row within the slice
  const unsigned row0 = DVW * slice + rloc;

  const int* anc_r = p.anc_rd + long(r) * wmax * tmax;
  const unsigned kslot = DK * IOB, vslot = DV * IOB;
  auto k_slab = [&](int j) {
    return static_cast<char*>(p.ak) + ((long(r) * tmax + j) * p.HK + hk) * wmax * long(kslot);
  };
  auto v_slab = [&](int j) {
    return static_cast<char*>(p.av) + ((long(r) * tmax + j) * p.HV + hv) * wmax * long(vslot);
  };
  auto d_slab = [&](int j) {  // delta rows use the input row size (fp16 / fp32)
    return static_cast<char*>(p.ad) + ((long(r) * tmax + j) * p.HV + hv) * wmax * long(vslot);
  };
  auto ab_slab = [&](int j) { return p.ab + ((long(r) * tmax + j) * p.HV + hv) * wmax; };
  auto ds_slab = [&](int j) { return p.adsc + ((long(r) * tmax + j) * p.HV + hv) * wmax; };

  // ---- round 1: indices, then query and the beam's step-t inputs.  Every
  // load is made by the fold lanes of the beam, as whole lines (see the
  // input-record kernel).
  int fsrc[NAX];
  bool fpok = true;
  int fpar = 0;
  if constexpr (NA > 0) {
    if constexpr (FUSED) {
      fpar = p.parents[long(r) * W + fbc];
    } else {
#pragma unroll
      for (int j = 0; j < NA; ++j) fsrc[j] = anc_r[fbc * tmax + j];
    }
  }
  // FUSED, t >= 2: the previous beams' ancestry rows staged in LDS by the
  // first four waves (as in the input-record kernel).
  const int ntab = kTab ? p.W_prev * (NA - 1) : 0;
  const bool tab = kTab && ntab <= kAncTable;
  int tv[kTab ? NTV : 1];
  if constexpr (kTab) {
    if (tab && tid < NL) {
#pragma unroll
      for (int i = 0; i < NTV; ++i)
        if (i * NL < ntab) {
          const int e = tid + NL * i;
          const int ec = e < ntab ? e : 0;
          const int pb = ec / (NA - 1);
          tv[i] = anc_r[pb * tmax + (ec - pb * (NA - 1))];
        }
    }
  }
  using K8 = RawV<BF16, 8>;
  using VR = RawV<BF16, RPL>;
  using VL = RawV<BF16, VPL>;
  K8 qr[C8], kt[C8];
  K8 kr[NAX][C8];
  float alr[NAX];
  unsigned esc[NAX];  // scale exponents of the ancestral delta rows (bf16 io)
  float2 abt;
  VL vt;
  VL dr[NAX];
  {
    const unsigned qoff = ((unsigned(r) * W + fbc) * p.HK + hk) * kslot + li * EPL * IOB;
#pragma unroll
    for (int c = 0; c < C8; ++c) qr[c].load(p.q, qoff + c * K8::kBytes);
    if constexpr (FUSED) {
#pragma unroll
      for (int c = 0; c < C8; ++c) kt[c].load(p.k_in, qoff + c * K8::kBytes);
      const unsigned gi = (unsigned(r) * W + fbc) * p.HV + hv;
      abt = make_float2(p.alpha_in[gi], p.beta_in[gi]);
      vt.load(p.v_in, gi * vslot + voff);
    } else {
      const char* ks = k_slab(NA);
#pragma unroll
      for (int c = 0; c < C8; ++c)
        kt[c].load(ks, fbc * kslot + li * EPL * IOB + c * K8::kBytes);
      abt = ab_slab(NA)[fbc];
      vt.load(v_slab(NA), fbc * vslot + voff);
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (kTab) {
    if (tab) {
      if (tid < NL) {
#pragma unroll
        for (int i = 0; i < NTV; ++i) {
          const int e = tid + NL * i;
          if (i * NL < ntab && e < ntab) anc_lds[e] = tv[i];
        }
      }
      __syncthreads();
    }
  }

  // ---- ancestral records: keys, decays and this lane's delta rows.  FUSED:
  // the parent's own step-(t-1) record first.
  bool fok[NAX];
  auto load_rec = [&](int j, int slot) {
    const char* ks = k_slab(j);
#pragma unroll
    for (int c = 0; c < C8; ++c) kr[j][c].load(ks, slot * kslot + li * EPL * IOB + c * K8::kBytes);
    alr[j] = ab_slab(j)[slot].x;
    if constexpr (BF16) esc[j] = ds_slab(j)[slot];
    dr[j].load(d_slab(j), slot * vslot + voff);
  };
  if constexpr (FUSED && NA > 0) {
    fpok = unsigned(fpar) < unsigned(p.W_prev);
    const int pf = fpok ? fpar : 0;
    fsrc[NA - 1] = pf;
    fok[NA - 1] = fpok;
    load_rec(NA - 1, pf);
    if (tab) {
#pragma unroll
      for (int j = 0; j < NA - 1; ++j) fsrc[j] = anc_lds[pf * (NA - 1) + j];
    } else {
#pragma unroll
      for (int j = 0; j < NA - 1; ++j) fsrc[j] = anc_r[pf * tmax + j];
      // wait inside the branch (see the input-record kernel)
      if constexpr (NA >= 2) __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < NA - 1; ++j) {
      fok[j] = fpok && unsigned(fsrc[j]) < unsigned(wmax);
      load_rec(j, fok[j] ? fsrc[j] : 0);
    }
  } else {
#pragma unroll
    for (int j = 0; j < NA; ++j) {
      fok[j] = unsigned(fsrc[j]) < unsigned(wmax);
      load_rec(j, fok[j] ? fsrc[j] : 0);
    }
  }

  // ---- shared-state rows (A fragments), as in the input-record kernel
  float4 Araw[NA == 0 ? KS : 1][MB][2];
  uint4 A[KS][MB][2];
  uint4* const frag =
      p.s_frag + ((long(unit) * NS + slice) * NW + w) * (KS * MB * 2 * 64) + lane;
  if constexpr (NA == 0) {
    const int m = lane & 15;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const unsigned row = DVW * slice + 16 * MB * w + 4 * MB * (m >> 2) + 4 * mb + (m & 3);
        const unsigned off = ((unsigned(unit) * DV + row) * DK + 32 * ks + 8 * (lane >> 4)) * 4u;
        Araw[ks][mb][0] = *at<float4>(p.s0, off);
        Araw[ks][mb][1] = *at<float4>(p.s0, off + 16);
      }
  } else {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int hl = 0; hl < 2; ++hl) A[ks][mb][hl] = frag[((ks * MB + mb) * 2 + hl) * 64];
  }
  __builtin_amdgcn_sched_barrier(0);

  // ---- phase 1: stage q_t and k_t as MFMA B fragments
  float qf[EPL], kf[EPL];
#pragma unroll
  for (int c = 0; c < C8; ++c) {
    qr[c].to_float(qf + 8 * c);
    kt[c].to_float(kf + 8 * c);
    const int k0 = li * EPL + 8 * c;
    uint4 hi, lo;
    split8(qf + 8 * c, hi, lo);
    b_lds[0][0][fb >> 4][k0 >> 5][(k0 >> 3) & 3][fb & 15] = hi;
    if constexpr (HL == 2) b_lds[0][1][fb >> 4][k0 >> 5][(k0 >> 3) & 3][fb & 15] = lo;
    split8(kf + 8 * c, hi, lo);
    b_lds[1][0][fb >> 4][k0 >> 5][(k0 >> 3) & 3][fb & 15] = hi;
    if constexpr (HL == 2) b_lds[1][1][fb >> 4][k0 >> 5][(k0 >> 3) & 3][fb & 15] = lo;
  }
  if constexpr (NA == 0) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const float x[8] = {Araw[ks][mb][0].x, Araw[ks][mb][0].y, Araw[ks][mb][0].z,
                            Araw[ks][mb][0].w, Araw[ks][mb][1].x, Araw[ks][mb][1].y,
                            Araw[ks][mb][1].z, Araw[ks][mb][1].w};
        split8(x, A[ks][mb][0], A[ks][mb][1]);
        if (tile == 0)
#pragma unroll
          for (int hl = 0; hl < 2; ++hl) frag[((ks * MB + mb) * 2 + hl) * 64] = A[ks][mb][hl];
      }
  }
  __syncthreads();

  // ---- phase 2: u_q = S_ctx q_t, u_k = S_ctx k_t on MFMA (no record needed)
  f32x4 accq[NBLK][MB], acck[NBLK][MB];
#pragma unroll
  for (int nb = 0; nb < NBLK; ++nb)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      accq[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
      acck[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
    for (int nb = 0; nb < NBLK; ++nb) {
      const uint4 bq = b_lds[0][0][nb][ks][g4][lane & 15];
      const uint4 bk = b_lds[1][0][nb][ks][g4][lane & 15];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        accq[nb][mb] = mfma_bf16(A[ks][mb][1], bq, accq[nb][mb]);
        acck[nb][mb] = mfma_bf16(A[ks][mb][1], bk, acck[nb][mb]);
        if constexpr (HL == 2) {
          const uint4 bql = b_lds[0][1][nb][ks][g4][lane & 15];
          const uint4 bkl = b_lds[1][1][nb][ks][g4][lane & 15];
          accq[nb][mb] = mfma_bf16(A[ks][mb][0], bql, accq[nb][mb]);
          acck[nb][mb] = mfma_bf16(A[ks][mb][0], bkl, acck[nb][mb]);
        }
        accq[nb][mb] = mfma_bf16(A[ks][mb][0], bq, accq[nb][mb]);
        acck[nb][mb] = mfma_bf16(A[ks][mb][0], bk, acck[nb][mb]);
      }
    }
  }

  // ---- phase 3: record dots and per-beam scalars (independent across j)
  {
    float c0 = 0.f, c1 = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; e += 2) {
      c0 = fmaf(kf[e], qf[e], c0);
      c1 = fmaf(kf[e + 1], qf[e + 1], c1);
    }
    const float cqt = group_sum<LPB>(c0 + c1);
    float cq[NAX], ck[NAX];
#pragma unroll
    for (int j = 0; j < NA; ++j) {
      float kj[EPL];
#pragma unroll
      for (int c = 0; c < C8; ++c) kr[j][c].to_float(kj + 8 * c);
      float a0 = 0.f, a1 = 0.f, b0v = 0.f, b1v = 0.f;
#pragma unroll
      for (int e = 0; e < EPL; e += 2) {
        a0 = fmaf(kj[e], qf[e], a0);
        a1 = fmaf(kj[e + 1], qf[e + 1], a1);
        b0v = fmaf(kj[e], kf[e], b0v);
        b1v = fmaf(kj[e + 1], kf[e + 1], b1v);
      }
      cq[j] = group_sum<LPB>(a0 + a1);
      ck[j] = group_sum<LPB>(b0v + b1v);
    }
    // the record terms of both projections over this lane's rows:
    // w_j = (k_j . x) * prod of the decays of records newer than j
    float rq[VPL], rk[VPL];
#pragma unroll
    for (int e = 0; e < VPL; ++e) rq[e] = rk[e] = 0.f;
    float decay = 1.f;
#pragma unroll
    for (int j = NA - 1; j >= 0; --j) {
      const float wq = fok[j] ? decay * cq[j] : 0.f, wk = fok[j] ? decay * ck[j] : 0.f;
      float dj[VPL];
      delta_to_float<BF16>(dr[j].w, dj, VPL);
      if constexpr (BF16) {
        const int e = int(static_cast<signed char>((esc[j] >> (8 * slice)) & 0xffu));
#pragma unroll
        for (int x = 0; x < VPL; ++x) dj[x] = ldexpf(dj[x], e);
      }
#pragma unroll
      for (int e = 0; e < VPL; ++e) {
        rq[e] = fmaf(wq, dj[e], rq[e]);
        rk[e] = fmaf(wk, dj[e], rk[e]);
      }
      decay *= fok[j] ? alr[j] : 1.f;
    }
    float vf[VPL];
    vt.to_float(vf);
#pragma unroll
    for (int e = 0; e < VPL; e += 4) {
      *reinterpret_cast<float4*>(&rq_lds[fb][li * VPL + e]) =
          make_float4(rq[e], rq[e + 1], rq[e + 2], rq[e + 3]);
      *reinterpret_cast<float4*>(&rk_lds[fb][li * VPL + e]) =
          make_float4(rk[e], rk[e + 1], rk[e + 2], rk[e + 3]);
      *reinterpret_cast<float4*>(&vt_lds[fb][li * VPL + e]) =
          make_float4(vf[e], vf[e + 1], vf[e + 2], vf[e + 3]);
    }
    if (li == 0) {
      sc_lds[fb][0] = decay;
      sc_lds[fb][1] = abt.x;
      sc_lds[fb][2] = abt.y;
      sc_lds[fb][3] = cqt;
    }
  }

  // ---- FUSED: index h_t and the step-t key and gates into the context
  if constexpr (FUSED) {
    if (fvalid && slice == 0) {
      if (hv == 0 && li == 0 && NA > 0) {
        int* dst = p.anc_wr + (long(r) * wmax + fbeam) * tmax;
        int* g = p.gather_out ? p.gather_out + (long(r) * W + fbeam) * NA : nullptr;
#pragma unroll
        for (int j = 0; j < NA; ++j) {
          const int h = fpok ? fsrc[j] : -1;
          dst[j] = h;
          if (g) g[j] = h;
        }
        if (!fpok) atomicOr(p.status, kStatusParent);
      }
      if (hv % p.G == 0) {
        char* ks = k_slab(NA);
#pragma unroll
        for (int c = 0; c < C8; ++c)
          kt[c].store(ks, fbeam * kslot + li * EPL * IOB + c * K8::kBytes);
      }
      if (li == 0) ab_slab(NA)[fbeam] = abt;
    }
  }
  __syncthreads();

  // ---- phase 4: Eq. 4 per output row; append delta_t
  __shared__ float mx_lds[NW][BEAMS];  // per wave and beam: largest |delta_t| of its rows
  float dts[NBLK][RPL];
#pragma unroll
  for (int nb = 0; nb < NBLK; ++nb) {
    const int bl = nb * 16 + (lane & 15);
    const int sb = b0 + bl;
    const float decay = sc_lds[bl][0], at_ = sc_lds[bl][1], bt = sc_lds[bl][2],
                cqt = sc_lds[bl][3];
    float uq[RPL], uk[RPL], vf[RPL];
#pragma unroll
    for (int e = 0; e < RPL; ++e) {
      uq[e] = fmaf(decay, accq[nb][e >> 2][e & 3], rq_lds[bl][rloc + e]);
      uk[e] = fmaf(decay, acck[nb][e >> 2][e & 3], rk_lds[bl][rloc + e]);
      vf[e] = vt_lds[bl][rloc + e];
    }
    float dt[RPL], ov[RPL];
#pragma unroll
    for (int e = 0; e < RPL; ++e) {
      dt[e] = bt * (vf[e] - at_ * uk[e]);
      ov[e] = fmaf(dt[e], cqt, at_ * uq[e]);
    }
    if (sb < W) {
      const unsigned ooff = (((unsigned(r) * W + sb) * p.HV + hv) * DV + row0) * 4u;
#pragma unroll
      for (int i = 0; i < MB; ++i)  // o is not read again: streaming stores
        store_out(p.o, ooff + 16u * i, f32x4{ov[4 * i], ov[4 * i + 1], ov[4 * i + 2], ov[4 * i + 3]});
    }
    float mx = 0.f;
#pragma unroll
    for (int e = 0; e < RPL; ++e) {
      dts[nb][e] = dt[e];
      mx = fmaxf(mx, fabsf(dt[e]));
    }
    if constexpr (BF16) {  // the beam's 4 lane groups of this wave, then the waves
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      if (g4 == 0) mx_lds[w][bl] = mx;
    }
  }
  if constexpr (BF16) __syncthreads();
#pragma unroll
  for (int nb = 0; nb < NBLK; ++nb) {
    const int bl = nb * 16 + (lane & 15);
    const int sb = b0 + bl;
    int e = 0;  // the slice's largest |delta_t| becomes 2^14 .. 2^15 (bf16 io)
    if constexpr (BF16) {
      float mx = 0.f;
#pragma unroll
      for (int w2 = 0; w2 < NW; ++w2) mx = fmaxf(mx, mx_lds[w2][bl]);
      int ex = 0;
      frexpf(mx, &ex);  // mx = f 2^ex, f in [0.5, 1)
      e = mx > 0.f ? ex - 15 : 0;
      e = e < -128 ? -128 : (e > 127 ? 127 : e);
    }
    if (sb < W) {
      float ds[RPL];
#pragma unroll
      for (int x = 0; x < RPL; ++x) ds[x] = BF16 ? ldexpf(dts[nb][x], -e) : dts[nb][x];
      VR dw;
      float_to_delta<BF16>(ds, dw.w, RPL);
      dw.store(d_slab(NA), sb * vslot + row0 * IOB);
      if constexpr (BF16)
        if (w == 0 && g4 == 0)
          reinterpret_cast<signed char*>(ds_slab(NA) + sb)[slice] = static_cast<signed char>(e);
    }
  }
}

template <int DK, int DV, int DVW, bool BF16, bool FUSED>
hipError_t launch_chain(int chain, const ReplayParams& prm, unsigned blocks, hipStream_t st) {
  constexpr int NBLK = kDecodeBeamBlocks;
  constexpr int threads = 4 * DK;
  switch (chain) {
#define ONELA_CHAIN_CASE(C)                                                              \
  case C:                                                                               \
    replay_kernel<DK, DV, DVW, NBLK, C, BF16, FUSED><<<blocks, threads, 0, st>>>(prm);  \
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

template <bool FUSED>
hipError_t launch_mode(const Shape& s, int step, const ReplayParams& prm, unsigned units,
                       hipStream_t st) {
  const int chain = step + 1;
#define ONELA_SHAPE(DK, DV, DVW)                                                          \
  if (s.dk == DK && s.dv == DV) {                                                        \
    const unsigned blocks = units * unsigned(DV / DVW) * unsigned(prm.ntiles);            \
    return s.bf16 ? launch_chain<DK, DV, DVW, true, FUSED>(chain, prm, blocks, st)      \
                  : launch_chain<DK, DV, DVW, false, FUSED>(chain, prm, blocks, st);    \
  }
#define ONELA_SHAPE_BF16(DK, DV, DVW)                                                     \
  if (s.dk == DK && s.dv == DV && s.bf16) {                                              \
    const unsigned blocks = units * unsigned(DV / DVW) * unsigned(prm.ntiles);            \
    return launch_chain<DK, DV, DVW, true, FUSED>(chain, prm, blocks, st);               \
  }
  ONELA_SHAPE(32, 32, 32)
  ONELA_SHAPE(64, 64, 64)
  ONELA_SHAPE(128, 128, 128)
  ONELA_SHAPE_BF16(128, 256, 256)
  ONELA_SHAPE_BF16(128, 512, 256)
  ONELA_SHAPE_BF16(256, 256, 256)
  ONELA_SHAPE_BF16(256, 512, 256)
#undef ONELA_SHAPE
#undef ONELA_SHAPE_BF16
  return hipErrorInvalidValue;
}

ReplayParams base_params(const Shape& s, int width, const void* q, float* o, const Arena& a,
                         unsigned* units_out) {
  constexpr int BEAMS = 16 * kDecodeBeamBlocks;
  ReplayParams prm = {};
  prm.q = q;
  prm.o = o;
  prm.s0 = a.s0;
  prm.s_frag = reinterpret_cast<uint4*>(a.s_frag);
  prm.ak = a.k;
  prm.av = a.v;
  prm.ab = a.ab;
  prm.ad = a.d;
  prm.adsc = a.dsc;
  prm.status = a.status;
  prm.R = s.R;
  prm.HK = s.HK;
  prm.HV = s.HV;
  prm.G = s.HV / s.HK;
  prm.W = width;
  prm.wmax = s.wmax;
  prm.tmax = s.tmax;
  prm.ntiles = (width + BEAMS - 1) / BEAMS;
  const int units = s.R * s.HV;
  prm.xcd_map = (units % 8 == 0) ? 1 : 0;
  *units_out = unsigned(units);
  return prm;
}

}  // namespace

hipError_t launch_replay_decode(const Shape& s, int step, int width, const void* q, float* o,
                                const Arena& a, hipStream_t st) {
  unsigned units;
  ReplayParams prm = base_params(s, width, q, o, a, &units);
  prm.anc_rd = a.anc[step & 1];
  return launch_mode<false>(s, step, prm, units, st);
}

hipError_t launch_replay_fused(const Shape& s, int step, int width, int prev_width,
                               const int* parents, const void* k, const void* v,
                               const float* alpha, const float* beta, const void* q, float* o,
                               int* gather_out, const Arena& a, hipStream_t st) {
  unsigned units;
  ReplayParams prm = base_params(s, width, q, o, a, &units);
  prm.parents = parents;
  prm.k_in = k;
  prm.v_in = v;
  prm.alpha_in = alpha;
  prm.beta_in = beta;
  prm.gather_out = gather_out;
  prm.W_prev = prev_width;
  prm.anc_rd = a.anc[(step + 1) & 1];
  prm.anc_wr = a.anc[step & 1];
  return launch_mode<true>(s, step, prm, units, st);
}

}  // namespace onela
