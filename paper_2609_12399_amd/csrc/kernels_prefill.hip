// Chunked prefill of the shared post-prefill state S_ctx (Sec. 3.1) on gfx950:
// Eq. 1 (Sec. 2.2) over a prompt, from S = 0, in chunks of C = 64 tokens.
//
// Inside a chunk that starts from state S_0, write Eq. 1 with the paper's
// correction term (Eq. 2), delta_t = beta_t (v_t - alpha_t S_{t-1} k_t), as
// S_t = alpha_t S_{t-1} + delta_t k_t^T.  Unrolling it with
// Gamma(t, i) = alpha_{i+1} ... alpha_t and gamma_t = Gamma(t, -1):
//   S_t     = gamma_t S_0 + sum_{i<=t} Gamma(t, i) delta_i k_i^T
//   delta_t = beta_t v_t - beta_t gamma_t S_0 k_t
//             - sum_{i<t} beta_t Gamma(t, i) (k_t . k_i) delta_i.
// With M the strictly lower C x C matrix M(t, i) = beta_t Gamma(t, i) (k_t.k_i)
// and T = (I + M)^{-1} (unit lower triangular), the deltas of the chunk are
//   D = U - W S_0^T,   U = T diag(beta) V,   W = T diag(beta gamma) K,
// and the state after the chunk is
//   S_C = g S_0 + D^T Kt,   Kt = diag(sigma) K,  sigma_t = Gamma(C - 1, t),
// g = gamma_{C-1}.  U, W and Kt depend only on the chunk's own tokens.  The
// workspace holds them as W' = diag(sigma) W, U' = diag(sigma) U and the plain
// keys K: with D' = diag(sigma) D = U' - W' S_0^T the update is
// S_C = g S_0 + D'^T K, and the keys keep their io encoding (bf16 keys are
// stored exactly, in half the bytes of fp32 sigma-scaled keys).
//
//   phase 1 (prefill_chunk_kernel): one workgroup per (request, value head,
//     chunk) forms the decay products Gamma from a doubling table (lane
//     shuffles), M from K K^T, T by forward substitution (each column held in
//     registers by a quad of lanes), then W and U, and stores W', K^T (io
//     dtype), U'^T and g to the workspace.  The
//     three products run on v_mfma_f32_16x16x4f32.  No division: products of
//     alpha are formed directly, so alpha = 0 is exact.  Each operand of
//     phase 2 is stored in the order phase 2's lanes load it (16 bytes per
//     lane, whole 1 KB blocks per wave); W' is formed transposed so that a
//     lane holds 4 consecutive keys of one token.
//   phase 2 (prefill_scan_kernel): one workgroup per (request, value head, 16
//     state rows; the row blocks of a head share one XCD) walks the chunks in
//     order: X^T = W' S^T, D'^T = U'^T - X^T, S^T <- g S^T + K^T D'^T, on
//     v_mfma_f32_16x16x4f32 (the update with bf16 keys on
//     v_mfma_f32_16x16x32_bf16, D' split exactly into three bf16 parts, so
//     that its products too are exact).  Wave w owns the state columns 16 w .. 16 w + 15
//     (a 16 x 16 fp32 accumulator tile that never leaves registers); the
//     contraction orders are chosen so that the tile is directly the B
//     operand of the next chunk's X and X's output is directly the B operand
//     of the update.  The partial X of the d_k / 16 waves are summed through
//     LDS, each token tile by d_k / 64 waves that take a share of its
//     accumulator components.
// A ragged last chunk is padded with alpha = 1, beta = 0, k = v = 0, which
// leaves the state unchanged.
#include <type_traits>

#include "device_common.h"
#include "internal.h"

namespace onela {
namespace {

constexpr int kC = kPrefillChunk;  // tokens per chunk
constexpr int kP1Threads = 256;

struct PrefillParams {
  const void* k;      // [R][P][HK][DK] io dtype
  const void* v;      // [R][P][HV][DV] io dtype
  const float* alpha; // [R][P][HV]
  const float* beta;
  float* s_out;       // [R][HV][DV][DK]
  // per (request, value head, chunk), in phase 2's fragment order:
  float* wb;          // [R*HV][nch][DK/16][4][64] f32x4   W' = diag(sigma) W
  void* ktb;          // [R*HV][nch] x DK*C keys, io dtype   K^T
  float* utb;         // [R*HV][nch][DV/16][4][64] f32x4   U'^T = (diag(sigma) U)^T
  float* gb;          // [R*HV][nch][16]  g, repeated (phase 2 loads it per lane)
  int HK, HV, P, nch;
  int xcd_map;  // phase 2: all row blocks of a unit on one XCD (units % 8 == 0)
};

// 8 consecutive io elements (16 B of bf16 or 32 B of fp32) at element i.
template <bool BF16>
struct Io8 {
  uint4 u[BF16 ? 1 : 2];
  __device__ void load(const void* base, long i) {
    if constexpr (BF16) {
      u[0] = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + i);
    } else {
      const uint4* q = reinterpret_cast<const uint4*>(static_cast<const float*>(base) + i);
      u[0] = q[0];
      u[1] = q[1];
    }
  }
  __device__ float get(int e) const {
    if constexpr (BF16) {
      const unsigned w = (&u[0].x)[e >> 1];
      return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
    } else {
      return __uint_as_float((&u[e >> 2].x)[e & 3]);
    }
  }
};

// Fills dst[t][c] (t < kC, c < NCOL, row stride LD) from rows of an io
// array (row t at element row0(t) + c0, zero for t >= n), scaled by
// scale(t).  Every thread issues all of its loads before its first store.
template <int NCOL, int LD, bool BF16, typename RowFn, typename ScaleFn>
__device__ inline void fill_rows(float* dst, const void* src, int n, int c0, RowFn&& row0,
                                 ScaleFn&& scale) {
  constexpr int NV = kC * NCOL / 8;  // 8-element vectors
  constexpr int PER = (NV + kP1Threads - 1) / kP1Threads;
  Io8<BF16> buf[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int vi = threadIdx.x + q * kP1Threads;
    const int t = vi / (NCOL / 8), c = (vi - t * (NCOL / 8)) * 8;
    if (vi < NV && t < n) buf[q].load(src, row0(t) + c0 + c);
  }
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int vi = threadIdx.x + q * kP1Threads;
    const int t = vi / (NCOL / 8), c = (vi - t * (NCOL / 8)) * 8;
    if (vi < NV) {
      const float sc = t < n ? scale(t) : 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) dst[t * LD + c + e] = t < n ? sc * buf[q].get(e) : 0.f;
    }
  }
}

// ---- phase 1 ----------------------------------------------------------------

// Rows are padded to a multiple of 4 words plus 4 (bf16 keys: 8 elements), so
// that the 16 rows x 4 columns an MFMA operand read touches fall in distinct
// banks.  bf16 keys stay in their encoding (exact, half the space), which lets
// two workgroups share a CU.
template <int DK, bool BF16>
struct P1Shared {
  using KT = typename std::conditional<BF16, uint16_t, float>::type;
  static constexpr int KLD = BF16 ? DK + 8 : DK + 4;
  KT K[kC][KLD];          // the chunk's keys (padding rows zero)
  float T[kC][kC + 4];    // (I + M)^{-1}
  union {
    float M[kC][kC + 4];  // until T is formed
    float X[kC][128 + 4]; // then a 128-column block of beta V (fp32 keys)
    uint16_t V[kC][128 + 8];  // or of V, raw (bf16)
  };
  float P[7][kC];         // P[k][t]: product of the 2^k decays ending at token t
  alignas(16) float al[kC], be[kC], gam[kC], sig[kC], bg[kC];  // bg = beta gamma
  __device__ float key(int t, int c) const {
    if constexpr (BF16) return __uint_as_float(unsigned(K[t][c]) << 16);
    else return K[t][c];
  }
};

// alpha_{i+1} ... alpha_t (t - i >= 0 factors; none: 1) from the doubling
// table, in blocks of 2^k decays, largest first.  Products only, so a zero
// decay gives an exact zero.
__device__ inline float decay(const float (&P)[7][kC], int t, int i) {
  float g = 1.f;
  int pos = t;
  const int L = t - i;
#pragma unroll
  for (int k = 6; k >= 0; --k)
    if ((L >> k) & 1) {
      g *= P[k][pos];
      pos -= 1 << k;
    }
  return g;
}

// Sum over the 4 lanes of a quad.
__device__ inline float quad_sum(float x) {
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0xB1,
                                                             0xF, 0xF, false));  // [1,0,3,2]
  x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x4E,
                                                             0xF, 0xF, false));  // [2,3,0,1]
  return x;
}

__device__ inline f32x4 mfma4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// bf16 inputs: the products of phase 1 run on v_mfma_f32_16x16x32_bf16 (lane l
// supplies A(l % 16, 8 (l / 16) + j) and B(8 (l / 16) + j, l % 16), j = 0..7,
// of each 32-deep step).  The keys and values are exact in bf16; the fp32
// factor built from T is split into three bf16 parts whose sum is exactly
// that factor, so every product is exact and only the fp32 accumulation
// rounds, as on the fp32 matrix instruction.

// Rows s0 .. s0 + 7 of column c of a row-major bf16 array (row stride ld), as
// one operand.
__device__ inline uint4 gather8(const uint16_t* a, int ld, int s0, int c) {
  unsigned u[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
    u[j] = unsigned(a[(s0 + 2 * j) * ld + c]) | (unsigned(a[(s0 + 2 * j + 1) * ld + c]) << 16);
  return make_uint4(u[0], u[1], u[2], u[3]);
}

// x = hi + mid + lo (8 floats, three bf16 vectors; exact for normal x).
__device__ inline void split3(const float* x, uint4& hi, uint4& mid, uint4& lo) {
  unsigned h[4], m[4], l[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    h[i] = pack_bf16x2(x[2 * i], x[2 * i + 1]);
    const float r0 = x[2 * i] - bf16_lo_to_float(h[i]);
    const float r1 = x[2 * i + 1] - bf16_hi_to_float(h[i]);
    m[i] = pack_bf16x2(r0, r1);
    l[i] = pack_bf16x2(r0 - bf16_lo_to_float(m[i]), r1 - bf16_hi_to_float(m[i]));
  }
  hi = make_uint4(h[0], h[1], h[2], h[3]);
  mid = make_uint4(m[0], m[1], m[2], m[3]);
  lo = make_uint4(l[0], l[1], l[2], l[3]);
}

// Row t, columns s0 .. s0 + 7 of T scaled per column by f, split in three.
__device__ inline void t_row_split(const float (&T)[kC][kC + 4], const float* f, int t, int s0,
                                   uint4& hi, uint4& mid, uint4& lo) {
  const f32x4 t0 = *reinterpret_cast<const f32x4*>(&T[t][s0]);
  const f32x4 t1 = *reinterpret_cast<const f32x4*>(&T[t][s0 + 4]);
  const f32x4 f0 = *reinterpret_cast<const f32x4*>(f + s0);
  const f32x4 f1 = *reinterpret_cast<const f32x4*>(f + s0 + 4);
  const f32x4 p0 = t0 * f0, p1 = t1 * f1;
  const float x[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
  split3(x, hi, mid, lo);
}

// The products of phase 1 run on v_mfma_f32_16x16x4f32 in 16 x 16 tiles: for
// D = A B, lane l supplies A(l % 16, k) and B(k, l % 16) with k = l / 16 of
// each 4-deep step and holds D(4 (l / 16) + r, l % 16), r = 0..3.
template <int DK, int DV, bool BF16>
__global__ __launch_bounds__(kP1Threads) void prefill_chunk_kernel(PrefillParams p) {
  extern __shared__ __align__(16) unsigned char smem[];
  using Sh = P1Shared<DK, BF16>;
  Sh& sh = *reinterpret_cast<Sh*>(smem);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l16 = lane & 15, l4 = lane >> 4;
  const int c = blockIdx.x % p.nch, unit = blockIdx.x / p.nch;
  const int r = unit / p.HV, hv = unit - r * p.HV, hk = hv / (p.HV / p.HK);
  const int t0 = c * kC;
  const int n = min(kC, p.P - t0);
  const long tok0 = long(r) * p.P + t0;

  if constexpr (BF16) {  // raw 16-byte copies of the key rows (zero past the prompt)
    constexpr int NV = kC * DK / 8, PER = (NV + kP1Threads - 1) / kP1Threads;
    uint4 buf[PER];
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int vi = tid + q * kP1Threads, t = vi / (DK / 8), cc = (vi - t * (DK / 8)) * 8;
      buf[q] = make_uint4(0u, 0u, 0u, 0u);
      if (vi < NV && t < n)
        buf[q] = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p.k) +
                                                 ((tok0 + t) * p.HK + hk) * DK + cc);
    }
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int vi = tid + q * kP1Threads, t = vi / (DK / 8), cc = (vi - t * (DK / 8)) * 8;
      if (vi < NV) *reinterpret_cast<uint4*>(&sh.K[t][cc]) = buf[q];
    }
  } else {
    fill_rows<DK, Sh::KLD, false>(&sh.K[0][0], p.k, n, 0,
                                  [&](int t) { return ((tok0 + t) * p.HK + hk) * DK; },
                                  [](int) { return 1.f; });
  }
  if (tid < kC) {
    const bool in = tid < n;
    const float al = in ? p.alpha[(tok0 + tid) * p.HV + hv] : 1.f;
    sh.al[tid] = al;
    sh.be[tid] = in ? p.beta[(tok0 + tid) * p.HV + hv] : 0.f;
    // doubling table of decay products (lane t of wave 0 holds token t)
    float v = al;
    sh.P[0][tid] = v;
#pragma unroll
    for (int k = 1; k < 7; ++k) {
      const float u = __shfl_up(v, 1 << (k - 1));
      if (tid >= (1 << (k - 1))) v *= u;
      sh.P[k][tid] = v;
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    // gamma_t = alpha_0 ... alpha_t; sigma_t = alpha_{t+1} ... alpha_{C-1}
    sh.gam[tid] = decay(sh.P, tid, -1);
    sh.sig[tid] = decay(sh.P, kC - 1, tid);
    sh.bg[tid] = sh.be[tid] * sh.gam[tid];
  }
  // M is zero above its diagonal 16 x 16 tiles (the product below fills the
  // rest)
  for (int e = tid; e < kC * kC; e += kP1Threads) {
    const int t = e / kC, i = e - t * kC;
    if ((i >> 4) > (t >> 4)) sh.M[t][i] = 0.f;
  }
  __syncthreads();
  // M(t, i) = beta_t Gamma(t, i) (k_t . k_i) for i < t, 0 for i >= t: the ten
  // tiles on or below the diagonal of K K^T
  for (int x = w; x < 10; x += 4) {
    const int a = (x >= 1) + (x >= 3) + (x >= 6), b = x - a * (a + 1) / 2;
    f32x4 acc;
    if constexpr (BF16) {  // two chains of 16 x 16 x 32 steps over the keys
      f32x4 acc2[2] = {};
#pragma unroll
      for (int ks = 0; ks < DK / 32; ++ks)
        acc2[ks & 1] = mfma_bf16(*reinterpret_cast<const uint4*>(&sh.K[16 * a + l16][32 * ks + 8 * l4]),
                                 *reinterpret_cast<const uint4*>(&sh.K[16 * b + l16][32 * ks + 8 * l4]),
                                 acc2[ks & 1]);
      acc = acc2[0] + acc2[1];
    } else {
      f32x4 acc4[4] = {};  // four independent chains over the key dimension
#pragma unroll 8
      for (int ks = 0; ks < DK / 4; ++ks)
        acc4[ks & 3] = mfma4(sh.key(16 * a + l16, 4 * ks + l4), sh.key(16 * b + l16, 4 * ks + l4),
                             acc4[ks & 3]);
      acc = (acc4[0] + acc4[1]) + (acc4[2] + acc4[3]);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int t = 16 * a + 4 * l4 + q, i = 16 * b + l16;
      const float g = decay(sh.P, t, i < t ? i : t);  // (no factor on or above the diagonal)
      sh.M[t][i] = i < t ? sh.be[t] * g * acc[q] : 0.f;
    }
  }
  __syncthreads();
  // T = (I + M)^{-1} by forward substitution, T(t, j) = -sum_{i<t} M(t, i)
  // T(i, j) for t > j: column j = 16 w + lane / 4 is held in registers by the
  // quad of lanes 4 (j % 16) .. + 3, lane sub summing the rows i = sub mod 4
  {
    const int j = 16 * w + (lane >> 2), sub = lane & 3;
    float x[kC / 4];
#pragma unroll
    for (int m = 0; m < kC / 4; ++m) x[m] = 0.f;
#pragma unroll
    for (int t = 0; t < kC; ++t) {
      float sp[4] = {0.f, 0.f, 0.f, 0.f};  // rows not computed yet hold 0
#pragma unroll
      for (int m = 0; m < (t + 3) / 4; ++m) sp[m & 3] = fmaf(sh.M[t][sub + 4 * m], x[m], sp[m & 3]);
      const float s = quad_sum((sp[0] + sp[1]) + (sp[2] + sp[3]));
      const float val = t == j ? 1.f : (t > j ? -s : 0.f);
      if (sub == (t & 3)) x[t >> 2] = val;
    }
#pragma unroll
    for (int m = 0; m < kC / 4; ++m) sh.T[sub + 4 * m][j] = x[m];
  }
  __syncthreads();

  const long cu = long(unit) * p.nch + c;
  // The three operands of phase 2 are stored in the order its lanes load them
  // (16 bytes per lane, 1 KB per wave and fragment).  K^T in the io dtype (the
  // keys' own bits: bf16 keys stay exact): fragment (column block b, token tile
  // a) of lane l holds K(t = 16 a + 4 (l / 16) + j, k = 16 b + l % 16), j =
  // 0..3; bf16 fragments of the tiles 2 h and 2 h + 1 are interleaved per lane.
  if constexpr (BF16) {
    uint4* kdst = reinterpret_cast<uint4*>(static_cast<uint16_t*>(p.ktb) + cu * DK * kC);
    for (int e = tid; e < DK / 16 * 2 * 64; e += kP1Threads) {
      const int l = e & 63, h = (e >> 6) & 1, b = e >> 7;
      const int kk = 16 * b + (l & 15), tt = 32 * h + 4 * (l >> 4);
      unsigned x[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int t = tt + 16 * (q >> 1) + 2 * (q & 1);
        x[q] = unsigned(sh.K[t][kk]) | (unsigned(sh.K[t + 1][kk]) << 16);
      }
      kdst[e] = make_uint4(x[0], x[1], x[2], x[3]);
    }
  } else {
    f32x4* kdst = reinterpret_cast<f32x4*>(static_cast<float*>(p.ktb) + cu * DK * kC);
    for (int e = tid; e < DK / 16 * 4 * 64; e += kP1Threads) {
      const int l = e & 63, a = (e >> 6) & 3, b = e >> 8;
      const int kk = 16 * b + (l & 15), t = 16 * a + 4 * (l >> 4);
      kdst[e] = f32x4{sh.K[t][kk], sh.K[t + 1][kk], sh.K[t + 2][kk], sh.K[t + 3][kk]};
    }
  }
  // W' = diag(sigma) T diag(beta gamma) K, formed transposed so that a lane
  // holds 4 consecutive keys of one token: fragment (b, a) of lane l holds
  // W'(t = 16 a + l % 16, k = 16 b + 4 (l / 16) + i), i = 0..3
  f32x4* wdst = reinterpret_cast<f32x4*>(p.wb + cu * kC * DK);
  // (T is lower triangular: row block a needs k < 16 (a + 1))
  constexpr int NBW = DK / 16;
  if constexpr (BF16) {
    // W^T(k, t) = sum_s K(s, k) (T diag(beta gamma))(t, s): 32-token steps
    // (the first covering rows a = 0, 1, the second a = 2, 3); the factor
    // is split once per row block and used for all of the wave's key blocks
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const int nks = (a + 2) / 2;
      uint4 fh[2], fm[2], fl[2];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
        if (ks < nks) t_row_split(sh.T, sh.bg, 16 * a + l16, 32 * ks + 8 * l4, fh[ks], fm[ks], fl[ks]);
      for (int b = w; b < NBW; b += 4) {
        f32x4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = c0, c2 = c0;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
          if (ks < nks) {
            const uint4 kf = gather8(&sh.K[0][0], Sh::KLD, 32 * ks + 8 * l4, 16 * b + l16);
            c2 = mfma_bf16(kf, fl[ks], c2);
            c1 = mfma_bf16(kf, fm[ks], c1);
            c0 = mfma_bf16(kf, fh[ks], c0);
          }
        wdst[(b * 4 + a) * 64 + lane] = sh.sig[16 * a + l16] * ((c2 + c1) + c0);
      }
    }
  } else {
    for (int x = w; x < 4 * NBW; x += 4) {
      const int a = x / NBW, b = x - a * NBW;
      f32x4 acc4[4] = {};
      for (int ks = 0; ks < 4 * (a + 1); ks += 4) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int kk = 4 * (ks + u) + l4;
          acc4[u] = mfma4(sh.be[kk] * sh.gam[kk] * sh.key(kk, 16 * b + l16), sh.T[16 * a + l16][kk],
                          acc4[u]);
        }
      }
      const f32x4 acc = (acc4[0] + acc4[1]) + (acc4[2] + acc4[3]);
      wdst[(b * 4 + a) * 64 + lane] = sh.sig[16 * a + l16] * acc;
    }
  }
  // U' = diag(sigma) T diag(beta) V, as U'^T fragments: fragment (row block rb,
  // token tile a) of lane l holds U'^T(16 rb + l % 16, t = 16 a + 4 (l / 16) + j),
  // j = 0..3
  f32x4* udst = reinterpret_cast<f32x4*>(p.utb + cu * DV * kC);
  constexpr int VC = DV < 128 ? DV : 128;  // V columns per block
  constexpr int NBU = VC / 16;
  for (int cb = 0; cb < DV; cb += VC) {
    if constexpr (BF16) {
      // raw 16-byte copies of the value rows (zero past the prompt)
      constexpr int NV = kC * VC / 8, PER = (NV + kP1Threads - 1) / kP1Threads;
      uint4 buf[PER];
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        const int vi = tid + q * kP1Threads, t = vi / (VC / 8), cc = (vi - t * (VC / 8)) * 8;
        buf[q] = make_uint4(0u, 0u, 0u, 0u);
        if (vi < NV && t < n)
          buf[q] = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p.v) +
                                                   ((tok0 + t) * p.HV + hv) * DV + cb + cc);
      }
#pragma unroll
      for (int q = 0; q < PER; ++q) {
        const int vi = tid + q * kP1Threads, t = vi / (VC / 8), cc = (vi - t * (VC / 8)) * 8;
        if (vi < NV) *reinterpret_cast<uint4*>(&sh.V[t][cc]) = buf[q];
      }
      __syncthreads();
      // U(t, d) = sum_s (T diag(beta))(t, s) V(s, d), the factor split once
      // per row block
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int nks = (a + 2) / 2;
        uint4 fh[2], fm[2], fl[2];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
          if (ks < nks) t_row_split(sh.T, sh.be, 16 * a + l16, 32 * ks + 8 * l4, fh[ks], fm[ks], fl[ks]);
        const f32x4 sg = *reinterpret_cast<const f32x4*>(&sh.sig[16 * a + 4 * l4]);
        for (int b = w; b < NBU; b += 4) {
          f32x4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = c0, c2 = c0;
#pragma unroll
          for (int ks = 0; ks < 2; ++ks)
            if (ks < nks) {
              const uint4 vf = gather8(&sh.V[0][0], 128 + 8, 32 * ks + 8 * l4, 16 * b + l16);
              c2 = mfma_bf16(fl[ks], vf, c2);
              c1 = mfma_bf16(fm[ks], vf, c1);
              c0 = mfma_bf16(fh[ks], vf, c0);
            }
          udst[((cb / 16 + b) * 4 + a) * 64 + lane] = sg * ((c2 + c1) + c0);
        }
      }
    } else {
      fill_rows<VC, 128 + 4, BF16>(&sh.X[0][0], p.v, n, cb,
                               [&](int t) { return ((tok0 + t) * p.HV + hv) * DV; },
                               [&](int t) { return sh.be[t]; });
      __syncthreads();
      for (int x = w; x < 4 * NBU; x += 4) {
        const int a = x / NBU, b = x - a * NBU;
        f32x4 acc4[4] = {};
        for (int ks = 0; ks < 4 * (a + 1); ks += 4) {
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int kk = 4 * (ks + u) + l4;
            acc4[u] = mfma4(sh.T[16 * a + l16][kk], sh.X[kk][16 * b + l16], acc4[u]);
          }
        }
        const f32x4 acc = (acc4[0] + acc4[1]) + (acc4[2] + acc4[3]);
        const f32x4 sg = *reinterpret_cast<const f32x4*>(&sh.sig[16 * a + 4 * l4]);
        udst[((cb / 16 + b) * 4 + a) * 64 + lane] = sg * acc;
      }
    }
    __syncthreads();
  }
  if (tid < 16) p.gb[cu * 16 + tid] = sh.gam[kC - 1];
}

// ---- phase 2 ----------------------------------------------------------------

// Operands of one chunk for one lane (see prefill_scan_kernel), loaded from
// the workspace's fragment order.  The keys stay in their io encoding until
// they are used, so that a load issued for a later chunk is not waited for
// early; bf16 keys of two token tiles share one 16-byte load.
template <bool BF16, int NU>
struct ScanOps {
  f32x4 w[4], u[NU];
  typename std::conditional<BF16, uint4, f32x4>::type k[BF16 ? 2 : 4];
  float g;
  __device__ float key(int mt, int j) const {
    if constexpr (BF16) {
      const uint4 q = k[mt >> 1];
      const unsigned h = (mt & 1) ? (j < 2 ? q.z : q.w) : (j < 2 ? q.x : q.y);
      return __uint_as_float((j & 1) ? (h & 0xffff0000u) : (h << 16));
    } else {
      return k[mt][j];
    }
  }
};

template <int N>
struct Vec {
  typedef float type __attribute__((ext_vector_type(N)));
};
template <>
struct Vec<1> {
  typedef float type;
};

// Components N g .. N g + N - 1 of v.
template <int N>
__device__ inline typename Vec<N>::type slice(const f32x4& v, int g) {
  if constexpr (N == 4) {
    return v;
  } else if constexpr (N == 2) {
    return g == 0 ? v.xy : v.zw;
  } else {
    return v[g];
  }
}

template <int DK, int DV, bool BF16>
__global__ __launch_bounds__(4 * DK) void prefill_scan_kernel(PrefillParams p) {
  constexpr int NW = DK / 16;  // waves: state columns 16 w .. 16 w + 15
  // The NW partial X^T of a token tile are summed by NW / 4 waves, each taking
  // NCP of the 4 accumulator components a lane holds (with fewer than 4 waves
  // a wave sums TPW whole tiles).
  constexpr int TPW = NW >= 4 ? 1 : 4 / NW;
  constexpr int NCP = NW >= 4 ? 16 / NW : 4;
  constexpr int NG = 4 / NCP;
  using VN = typename Vec<NCP>::type;
  // operand sets in flight: three, two where three do not fit in the registers
  // of a 1024-thread workgroup
  constexpr int NS = (DK == 256 && !BF16) ? 2 : 3;
  __shared__ VN xp[NW][4][NG][64];  // partial X^T tiles of every wave, by component group
  __shared__ f32x4 ds[4][64];       // D'^T tiles: U'^T minus the sums of the partials
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  // The DV / 16 row blocks of a (request, value head) read the same W and
  // Kt of every chunk.  Workgroups are dispatched round-robin over the 8
  // XCDs (block i on XCD i % 8), so when the unit count is a multiple of 8
  // all row blocks of a unit are placed on one XCD and share its L2.
  constexpr int NRB = DV / 16;
  int rb, unit;
  if (p.xcd_map) {
    const int x = blockIdx.x & 7, slot = blockIdx.x >> 3;
    unit = x + 8 * (slot / NRB);
    rb = slot % NRB;
  } else {
    rb = blockIdx.x % NRB;
    unit = blockIdx.x / NRB;
  }
  const int row0 = 16 * rb;
  const int lr = lane & 15, lq = lane >> 4;
  // st[i] = S^T(k = 16 w + 4 lq + i, n = lr) = S(row0 + lr, 16 w + 4 lq + i)
  f32x4 st = {0.f, 0.f, 0.f, 0.f};
  float* dst = p.s_out + (long(unit) * DV + row0 + lr) * DK + 16 * w + 4 * lq;
  if (p.nch == 0) {  // empty prompt: S = 0, and there is no chunk to read
    *reinterpret_cast<f32x4*>(dst) = st;
    return;
  }
  // the token tiles whose D' this wave forms, and its component group
  const int g0 = NW >= 4 ? w >> 2 : 0;
  auto tile = [&](int i) { return NW >= 4 ? (w & 3) : w + NW * i; };
  // Loads are unconditional (past the end they re-read the last chunk) so
  // the compiler can count them and wait only for the set about to be used.
  // Every load is one lane's 16 bytes of a fragment stored contiguously by
  // phase 1, so a wave reads whole 1 KB blocks.
  auto load = [&](int c, ScanOps<BF16, TPW>& o) {
    const long cu = long(unit) * p.nch + (c < p.nch ? c : p.nch - 1);
    const f32x4* wc = reinterpret_cast<const f32x4*>(p.wb + cu * kC * DK);
    const f32x4* ut = reinterpret_cast<const f32x4*>(p.utb + cu * DV * kC);
    // g through the vector memory path (16 copies, one per lane of a row):
    // a scalar load would be waited for by the step's first LDS wait
    o.g = p.gb[cu * 16 + lr];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) o.w[mt] = wc[(w * 4 + mt) * 64 + lane];
    if constexpr (BF16) {
      const uint4* kt = reinterpret_cast<const uint4*>(static_cast<const __bf16*>(p.ktb) +
                                                       cu * DK * kC);
#pragma unroll
      for (int h = 0; h < 2; ++h) o.k[h] = kt[(w * 2 + h) * 64 + lane];
    } else {
      const f32x4* kt = reinterpret_cast<const f32x4*>(static_cast<const float*>(p.ktb) +
                                                       cu * DK * kC);
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) o.k[mt] = kt[(w * 4 + mt) * 64 + lane];
    }
#pragma unroll
    for (int i = 0; i < TPW; ++i) o.u[i] = ut[(rb * 4 + tile(i)) * 64 + lane];
  };
  auto step = [&](int c, const ScanOps<BF16, TPW>& o) {
    if (c >= p.nch) return;
    // partial X^T(t, n) over this wave's 16 state columns: four independent
    // accumulator chains, one per token tile
    f32x4 xa[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) xa[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
        xa[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.w[mt][i], st[i], xa[mt], 0, 0, 0);
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int g = 0; g < NG; ++g) xp[w][mt][g][lane] = slice<NCP>(xa[mt], g);
    __syncthreads();
    // D'^T(t = 16 mt + 4 lq + j, n = lr) = U'^T - sum over the waves of X^T,
    // components NCP g0 .. of the tiles this wave forms
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
      const int mt = tile(i);
      VN x = xp[0][mt][g0][lane];
#pragma unroll
      for (int v = 1; v < NW; ++v) x += xp[v][mt][g0][lane];
      *reinterpret_cast<VN*>(reinterpret_cast<float*>(&ds[mt][lane]) + NCP * g0) =
          slice<NCP>(o.u[i], g0) - x;
    }
    __syncthreads();
    // S^T <- g S^T + K^T D'^T
    f32x4 sum;
    if constexpr (BF16) {
      // on v_mfma_f32_16x16x32_bf16, two token tiles per 32-deep step: the
      // step's k = 8 lq + i stands for token 16 (2 h + i / 4) + 4 lq + i % 4,
      // so that the lane's keys are its 16-byte load as it stands and its D'
      // values are its own components of the two tiles.  The keys are exact
      // in bf16 and D' is split exactly into three bf16 parts, so every
      // product is exact and only the fp32 accumulation rounds.
      f32x4 up[2], uq[2], ur[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const f32x4 d0 = ds[2 * h][lane], d1 = ds[2 * h + 1][lane];
        const float x[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
        uint4 dh, dm, dl;
        split3(x, dh, dm, dl);
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        up[h] = mfma_bf16(o.k[h], dh, z);
        uq[h] = mfma_bf16(o.k[h], dm, z);
        ur[h] = mfma_bf16(o.k[h], dl, z);
      }
      sum = (up[0] + up[1]) + ((uq[0] + uq[1]) + (ur[0] + ur[1]));
    } else {
      // one fp32 chain per token tile, summed
      f32x4 up[4], dd[4];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        dd[mt] = ds[mt][lane];
        up[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
          up[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.key(mt, j), dd[mt][j], up[mt], 0, 0, 0);
      sum = (up[0] + up[1]) + (up[2] + up[3]);
    }
    st = o.g * st + sum;
  };
  // NS operand sets in flight: chunk c + NS - 1 is requested before chunk c
  // is processed.  (xp and ds are rewritten only after the next chunk's first
  // barrier, which every wave reaches after reading them.)  The scheduling
  // barriers keep every load group in program order, so the wait before a
  // step covers only its own (oldest) group.
  ScanOps<BF16, TPW> a, b;
  if constexpr (NS == 3) {
    ScanOps<BF16, TPW> c3;
    load(0, a);
    __builtin_amdgcn_sched_barrier(0);
    load(1, b);
    for (int c = 0; c < p.nch; c += 3) {
      __builtin_amdgcn_sched_barrier(0);
      load(c + 2, c3);
      __builtin_amdgcn_sched_barrier(0);
      step(c, a);
      __builtin_amdgcn_sched_barrier(0);
      load(c + 3, a);
      __builtin_amdgcn_sched_barrier(0);
      step(c + 1, b);
      __builtin_amdgcn_sched_barrier(0);
      load(c + 4, b);
      __builtin_amdgcn_sched_barrier(0);
      step(c + 2, c3);
    }
  } else {
    load(0, a);
    for (int c = 0; c < p.nch; c += 2) {
      __builtin_amdgcn_sched_barrier(0);
      load(c + 1, b);
      __builtin_amdgcn_sched_barrier(0);
      step(c, a);
      __builtin_amdgcn_sched_barrier(0);
      load(c + 2, a);
      __builtin_amdgcn_sched_barrier(0);
      step(c + 1, b);
    }
  }
  *reinterpret_cast<f32x4*>(dst) = st;
}

template <int DK, int DV, bool BF16>
hipError_t launch_t(const Shape& s, const PrefillParams& prm, hipStream_t st) {
  const unsigned units = unsigned(s.R * s.HV);
  const size_t lds = sizeof(P1Shared<DK, BF16>);
  auto k1 = prefill_chunk_kernel<DK, DV, BF16>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k1),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  if (e != hipSuccess) return e;
  if (prm.nch > 0) {  // an empty prompt leaves S = 0 (phase 2 stores zeros)
    k1<<<units * unsigned(prm.nch), kP1Threads, lds, st>>>(prm);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  prefill_scan_kernel<DK, DV, BF16><<<units * unsigned(DV / 16), 4 * DK, 0, st>>>(prm);
  return hipGetLastError();
}

}  // namespace


hipError_t launch_prefill_chunked(const Shape& s, int prompt_len, const void* k, const void* v,
                                  const float* alpha, const float* beta, float* s0_out,
                                  void* workspace, hipStream_t st) {
  PrefillParams prm{};
  prm.k = k;
  prm.v = v;
  prm.alpha = alpha;
  prm.beta = beta;
  prm.s_out = s0_out;
  prm.HK = s.HK;
  prm.HV = s.HV;
  prm.P = prompt_len;
  prm.nch = (prompt_len + kC - 1) / kC;
  const size_t units = size_t(s.R) * s.HV, nch = size_t(prm.nch);
  prm.xcd_map = units % 8 == 0 ? 1 : 0;
  float* base = static_cast<float*>(workspace);
  prm.wb = base;
  float* const kt_base = prm.wb + units * nch * kC * s.dk;  // K^T region (fp32-sized)
  prm.ktb = kt_base;
  prm.utb = kt_base + units * nch * kC * s.dk;
  auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
  prm.gb = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                    up(units * nch * size_t(kC) * (2 * s.dk + s.dv) * 4));
#define ONELA_PF_SHAPE(DK, DV)                                                            \
  if (s.dk == DK && s.dv == DV)                                                         \
    return s.bf16 ? launch_t<DK, DV, true>(s, prm, st) : launch_t<DK, DV, false>(s, prm, st);
  ONELA_PF_SHAPE(32, 32)
  ONELA_PF_SHAPE(64, 64)
  ONELA_PF_SHAPE(128, 128)
  ONELA_PF_SHAPE(128, 256)
  ONELA_PF_SHAPE(128, 512)
  ONELA_PF_SHAPE(256, 256)
  ONELA_PF_SHAPE(256, 512)
#undef ONELA_PF_SHAPE
  return hipErrorInvalidValue;
}

}  // namespace onela
