// Large-beam GDN decode step for gfx950 (CDNA4).
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
// gives S_{t,b} q exactly (in exact arithmetic).  The fold is carried in
// scaled form p = s p~ with s the running product of the alphas, so each
// step costs one dot product and one axpy per element (p~ -= beta_j c~ k_j,
// c~ = k_j . p~, g_j = s beta_j c~, s *= alpha_j; alpha_j = 0 simply zeroes
// s).  The only d_v x d_k work is the final S_ctx p, a dense GEMM over all
// beams of a head, O_h = S_ctx[h] . [p_1 .. p_W], which runs on MFMA; the
// fold and the v-terms are vector work with 16-byte loads.
//
// Precision.  S_ctx (fp32) and p are split into bf16 hi + lo
// (hi = bf16(x), lo = bf16(x - hi)), and O = S_hi P_hi + S_hi P_lo + S_lo P_hi is
// accumulated in fp32 by v_mfma_f32_16x16x32_bf16 (about 16 significant bits
// per product; the dropped S_lo P_lo term is ~2^-17 relative).
//
// Work decomposition.  One workgroup = (request, value head, row slice of DVW
// state rows, 16*NBLK beams), min(d_k, DVW)/16 waves of 16*MB rows each
// (MB = DVW/d_k when DVW >= d_k, else 1; wide d_v and d_k = 256 are split into
// row slices, each folding its beams again).
// Phase 1 (fold): LPB lanes per beam, each owning EPL consecutive key
// elements and VPL = DVW/LPB consecutive value rows of its beam; dot products
// are reduced across those lanes with DPP, and each lane accumulates
// sum_j g_j v_j over its value rows as the g_j appear.  The folded queries
// are written, split into hi/lo, to LDS directly in MFMA B-fragment order,
// the value-term sums to LDS rows per beam.  Phase 2 (contract): wave w
// multiplies its 16*MB state rows (A fragments: split in registers from fp32
// S_ctx at step 0, stored split in the workspace for later steps) by the
// beams' B fragments, one 16-beam block at a time.  Phase 3 (epilogue),
// after each block's products: each lane holds 4*MB consecutive output rows
// of one beam, adds the value-term sums of those rows from LDS and stores
// them as 16-byte vectors.
//
// Every global load is made by the fold lane that owns the beam: whole
// 128-byte lines of q, k and v per record, plus one parent index and one
// ancestry row per beam.  A CU has a limited number of memory requests in
// flight, so the number of requests per wave, not only the bytes, sets how
// soon the second wave of each SIMD gets its data.
//
// Why 32 beams and 16 rows per wave: every workgroup streams its head's
// whole shared state (64 KiB at d = 128) through the CU's vector memory pipe
// as MFMA A fragments, which is most of a CU's traffic; one 512-thread
// workgroup per CU covering 32 beams moves half the state bytes per beam of
// two 16-beam workgroups at the same occupancy.
//
// Two modes share the kernel.  DECODE reads h_t and the step-t records from
// the context (after onela_resolve_ancestry and onela_append_records).
// FUSED performs the whole step in one launch: it reads the parents and the
// previous index h_{t-1} (Eq. 5: h_t(b, j) = h_{t-1}(pi(b), j), h_t(b, t-1) =
// pi(b)), reads the step-t records from the caller's buffers, writes them
// into the arena slab t (workgroups of value head 0 write h_t, those of the
// first value head of each group write k), and decodes.
//
// Loads are issued in the order they are waited for (the vector memory
// counter retires in order): indices first, then everything that does not
// depend on them, then the ancestral records once the indices are back.
//
// Block order is XCD-aware: workgroups are dispatched round-robin over the 8
// XCDs, so block id i runs on XCD i % 8; all beam tiles of a (request, head)
// are mapped to one XCD so that head's shared state and records stay in that
// XCD's L2.
#include "device_common.h"
#include "internal.h"

namespace onela {
namespace {


struct DecodeParams {
  const void* q;
  float* o;
  // FUSED only: the step's inputs from the caller
  const int* parents;
  const void* k_in;
  const void* v_in;
  const float* alpha_in;
  const float* beta_in;
  int* gather_out;
  int* status;
  // context
  const float* s0;  // shared state S_ctx, fp32 [R*HV][DV][DK] (read at step 0)
  uint4* s_frag;    // S_ctx split into bf16 hi/lo, A-fragment order (written at step 0)
  void* ak;
  void* av;
  // borrowed records: per-step caller buffers (see Arena); borrow != 0 selects them
  int borrow;
  const void* bk[kMaxSteps];
  const void* bv[kMaxSteps];
  const float* balpha[kMaxSteps];
  const float* bbeta[kMaxSteps];
  int bw[kMaxSteps];
  float2* ab;
  const int* anc_rd;  // h_t (DECODE) or h_{t-1} (FUSED)
  int* anc_wr;        // FUSED: h_t
  int R, HK, HV, G, W, W_prev, wmax, tmax;
  int ntiles;   // beam tiles per (request, value head)
  int xcd_map;  // 1: XCD-aware block order (units % 8 == 0)
};

// Threads of a decode workgroup covering DVW state rows at key dimension DK:
// one wave per 16*MB rows.
constexpr int decode_rows_per_wave(int dk, int dvw) { return 16 * (dvw >= dk ? dvw / dk : 1); }
constexpr int decode_threads(int dk, int dvw) { return 64 * (dvw / decode_rows_per_wave(dk, dvw)); }

template <int DK, int DV, int DVW, int NBLK, int CHAIN, bool BF16, bool FUSED, bool BORROW>
__global__ __launch_bounds__(decode_threads(DK, DVW)) void decode_kernel(DecodeParams p) {
  constexpr int MB = decode_rows_per_wave(DK, DVW) / 16;  // 16-row MFMA blocks per wave
  constexpr int NS = DV / DVW;       // row slices (workgroups) per (request, head, tile)
  constexpr int NW = DVW / (16 * MB);// waves per workgroup (= min(DK, DVW) / 16)
  constexpr int RPL = 4 * MB;        // consecutive output rows per epilogue lane
  static_assert((DVW >= DK ? MB * DK == DVW : DVW % 16 == 0) && NS * DVW == DV &&
                    (MB == 1 || MB == 2 || MB == 4),
                "state rows per workgroup: 1, 2 or 4 times d_k, or 16-row blocks below d_k");
  constexpr int NT = NW * 64;        // threads per workgroup
  constexpr int BEAMS = 16 * NBLK;   // beams per workgroup
  constexpr int LPB = NT / BEAMS;    // fold lanes per beam
  constexpr int EPL = DK / LPB;      // key elements per fold lane
  constexpr int C8 = EPL / 8;        // 8-element chunks per fold lane
  constexpr int VPL = DVW / LPB;     // value rows per fold lane
  constexpr int VS = DVW + 4;        // padded LDS row of the value-term sums
  constexpr int KS = DK / 32;        // MFMA k-steps
  constexpr int NA = CHAIN - 1;      // ancestral records (= step t)
  constexpr int NAX = NA > 0 ? NA : 1;
  constexpr unsigned IOB = BF16 ? 2 : 4;
  static_assert(EPL % 8 == 0 && EPL >= 8, "fold lanes must own 8-element chunks");
  static_assert(VPL == 8 || VPL == 16, "fold lanes own 8 or 16 value rows");
  static_assert(LPB <= 64 && (LPB & (LPB - 1)) == 0, "fold lane group within a wave");

  __shared__ uint4 p_lds[2][NBLK][KS][4][16];  // folded queries, B-fragment order
  __shared__ float v_lds[BEAMS][VS];           // sum_j g_j v_j per beam, this slice's rows
  // FUSED, t >= 2: columns 0..t-2 of the request's h_{t-1}, all previous beams
  constexpr bool kTab = FUSED && NA >= 2;
  constexpr int NL = NT < 256 ? NT : 256;      // table-loading threads (at most 4 waves)
  constexpr int NTV = kAncTable / NL;          // table entries per loading lane
  __shared__ int anc_lds[kTab ? kAncTable : 1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;

  // The arguments the first loads depend on, in scalar registers together:
  // left alone, the compiler loads each in the basic block that first uses
  // it, and the first memory requests wait for several dependent rounds of
  // argument loads (about 0.2 us each).
  // Fused with borrowed records: also the record pointers of the three
  // latest ancestral steps (and with them the argument cache lines of the
  // older ones), needed as soon as the parent is known.
  constexpr int J1 = NA > 0 ? NA - 1 : 0, J2 = NA > 1 ? NA - 2 : J1, J3 = NA > 2 ? NA - 3 : J2;
  if constexpr (FUSED && BORROW && NA > 0)
    asm volatile("" ::"s"(p.ntiles), "s"(p.xcd_map), "s"(p.HK), "s"(p.HV), "s"(p.G), "s"(p.W),
                 "s"(p.wmax), "s"(p.tmax), "s"(p.anc_rd), "s"(p.q), "s"(p.W_prev), "s"(p.parents),
                 "s"(p.k_in), "s"(p.v_in), "s"(p.alpha_in), "s"(p.beta_in), "s"(p.bk[J1]),
                 "s"(p.bv[J1]), "s"(p.balpha[J1]), "s"(p.bbeta[J1]), "s"(p.bk[J2]), "s"(p.bv[J2]),
                 "s"(p.balpha[J2]), "s"(p.bbeta[J2]), "s"(p.bk[J3]), "s"(p.bv[J3]),
                 "s"(p.balpha[J3]), "s"(p.bbeta[J3]));
  else if constexpr (FUSED)
    asm volatile("" ::"s"(p.ntiles), "s"(p.xcd_map), "s"(p.HK), "s"(p.HV), "s"(p.G), "s"(p.W),
                 "s"(p.wmax), "s"(p.tmax), "s"(p.anc_rd), "s"(p.q), "s"(p.W_prev), "s"(p.parents),
                 "s"(p.k_in), "s"(p.v_in), "s"(p.alpha_in), "s"(p.beta_in), "s"(p.anc_wr));
  else if constexpr (BORROW)
    asm volatile("" ::"s"(p.ntiles), "s"(p.xcd_map), "s"(p.HK), "s"(p.HV), "s"(p.G), "s"(p.W),
                 "s"(p.wmax), "s"(p.tmax), "s"(p.anc_rd), "s"(p.q), "s"(p.bk[NA]),
                 "s"(p.bv[NA]), "s"(p.balpha[NA]), "s"(p.bbeta[NA]), "s"(p.bw[NA]));
  else
    asm volatile("" ::"s"(p.ntiles), "s"(p.xcd_map), "s"(p.HK), "s"(p.HV), "s"(p.G), "s"(p.W),
                 "s"(p.wmax), "s"(p.tmax), "s"(p.anc_rd), "s"(p.q), "s"(p.ak), "s"(p.av),
                 "s"(p.ab));

  // A new beam search starts at step 0: no parent can be flagged yet, so the
  // step-0 launch zeroes the sticky status word.
  if constexpr (NA == 0) {
    if (blockIdx.x == 0 && tid == 0) p.status[0] = 0;
  }

  // block -> (unit = request*HV + head, row slice, beam tile); all slices and
  // tiles of a unit share an XCD when the unit count is a multiple of 8
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

  // fold lanes: beam fb of the tile, key elements [li*EPL, li*EPL + EPL) and
  // value rows DVW*slice + [li*VPL, li*VPL + VPL)
  const int fb = tid / LPB;
  const int li = tid - fb * LPB;
  const int fbeam = b0 + fb;
  const bool fvalid = fbeam < W;
  const int fbc = fvalid ? fbeam : 0;
  const unsigned voff = (unsigned(DVW) * slice + unsigned(li) * VPL) * IOB;
  // epilogue lanes: beam (lane & 15) of block nb, rows row0 + [0, RPL)
  const int g4 = lane >> 4;
  const unsigned rloc = 16 * MB * w + RPL * g4;  // row within the slice
  const unsigned row0 = DVW * slice + rloc;

  // uniform bases (per workgroup)
  const int* anc_r = p.anc_rd + long(r) * wmax * tmax;
  const unsigned kslot = DK * IOB, vslot = DV * IOB;
  // Record rows of step j: slot s of (r, j, head) at slab(j) + s * stride.
  // Arena: head-major slabs, stride one row.  Borrowed: the caller's step-j
  // buffers, beam-major, stride one beam.  The storage is a template
  // parameter so that each record's addresses are straight-line code, whose
  // argument loads the compiler issues in one round.
  constexpr bool borrow = BORROW;
  const unsigned kstride = borrow ? unsigned(p.HK) * kslot : kslot;
  const unsigned vstride = borrow ? unsigned(p.HV) * vslot : vslot;
  auto k_slab = [&](int j) -> char* {
    if constexpr (borrow)
      return const_cast<char*>(static_cast<const char*>(p.bk[j])) +
             (long(r) * p.bw[j] * p.HK + hk) * long(kslot);
    return static_cast<char*>(p.ak) + ((long(r) * tmax + j) * p.HK + hk) * wmax * long(kslot);
  };
  auto v_slab = [&](int j) -> char* {
    if constexpr (borrow)
      return const_cast<char*>(static_cast<const char*>(p.bv[j])) +
             (long(r) * p.bw[j] * p.HV + hv) * long(vslot);
    return static_cast<char*>(p.av) + ((long(r) * tmax + j) * p.HV + hv) * wmax * long(vslot);
  };
  auto ab_slab = [&](int j) { return p.ab + ((long(r) * tmax + j) * p.HV + hv) * wmax; };
  // slot bound of step j's records (borrowed buffers hold exactly w[j] beams)
  auto slot_ok = [&](int j, int sl) {
    if constexpr (borrow) return unsigned(sl) < unsigned(p.bw[j]);
    return unsigned(sl) < unsigned(wmax);
  };
  auto load_ab = [&](int j, int slot) -> float2 {
    if constexpr (borrow) {
      const long i = (long(r) * p.bw[j] + slot) * p.HV + hv;
      return make_float2(p.balpha[j][i], p.bbeta[j][i]);
    }
    return ab_slab(j)[slot];
  };

  // ---- round 1: indices (the parent in FUSED mode, the beam's row of h_t
  // otherwise), then every load that needs no index: the query and the
  // beam's own step-t record.  Each fold lane loads only its own beam's
  // data, as whole 128-byte lines, which keeps the number of memory
  // requests per wave small: a CU holds a limited number in flight, and
  // requests beyond it wait for earlier ones to return.
  int fsrc[NAX];
  bool fpok = true;
  int fpar = 0;
  // FUSED with 4 beams per wave (d_k = 128): the wave's 4 parents come in
  // one scalar load from the constant address space (the parents are only
  // read), which travels outside the vector memory queue: it is not held
  // behind the bulk loads the waves issue next, and arrives about 0.2 us
  // earlier at t = 1.  Each lane picks its beam's parent only where the
  // parent is first needed, so that nothing waits for it before the bulk
  // loads are issued.  A wave whose 4 beams are not all live (ragged last
  // tile) loads per lane as the other shapes do.
  typedef int i32x4 __attribute__((ext_vector_type(4)));
  i32x4 spv = {0, 0, 0, 0};
  constexpr bool kScalarPar = FUSED && NA > 0 && LPB == 16;
  bool spar = false;
  if constexpr (NA > 0) {
    if constexpr (FUSED) {
      if constexpr (kScalarPar) {
        const int wb = __builtin_amdgcn_readfirstlane(b0 + 4 * w);
        spar = wb + 4 <= W;
        if (spar) {
          typedef const __attribute__((address_space(4))) i32x4 ci32x4;
          spv = *(ci32x4*)(p.parents + (long(r) * W + wb));
        } else {
          fpar = p.parents[long(r) * W + fbc];
        }
      } else {
        fpar = p.parents[long(r) * W + fbc];
      }
    } else {
#pragma unroll
      for (int j = 0; j < NA; ++j) fsrc[j] = anc_r[fbc * tmax + j];
    }
  }
  // FUSED, t >= 2: the ancestry rows of all previous beams (their first t-1
  // entries, when they fit kAncTable) are loaded by the first four waves
  // right behind the parent indices and staged in LDS, so that the records
  // of steps <= t-2 are addressed as soon as a beam's parent is known rather
  // than one dependent memory round trip later.  Only the first wave of each
  // SIMD loads: the second receives its data about one round trip later.
  // Every workgroup loads its request's whole table, so the table's cost
  // grows with its size while what it saves (one dependent round) does not:
  // from chains of 5 (t >= 4) on, tables beyond 1024 entries are read row by
  // row (at 4 requests x 512 beams: 22.6 -> 20.2 us at t = 4).
  const int ntab = kTab ? p.W_prev * (NA - 1) : 0;
  const bool tab = kTab && ntab <= (NA >= 4 ? kAncTableLong : kAncTable);
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
  using VR = RawV<BF16, VPL>;
  K8 qr[C8];
  K8 kr[CHAIN][C8];
  float2 abr[CHAIN];
  VR vr[CHAIN];
  {
    const unsigned qoff = ((unsigned(r) * W + fbc) * p.HK + hk) * kslot + li * EPL * IOB;
#pragma unroll
    for (int c = 0; c < C8; ++c) qr[c].load(p.q, qoff + c * K8::kBytes);
    if constexpr (FUSED) {
#pragma unroll
      for (int c = 0; c < C8; ++c) kr[NA][c].load(p.k_in, qoff + c * K8::kBytes);
      const unsigned gi = (unsigned(r) * W + fbc) * p.HV + hv;
      abr[NA] = make_float2(p.alpha_in[gi], p.beta_in[gi]);
      vr[NA].load(p.v_in, gi * vslot + voff);
    } else {
      const char* ks = k_slab(NA);
#pragma unroll
      for (int c = 0; c < C8; ++c)
        kr[NA][c].load(ks, fbc * kstride + li * EPL * IOB + c * K8::kBytes);
      abr[NA] = load_ab(NA, fbc);
      vr[NA].load(v_slab(NA), fbc * vstride + voff);
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

  // ---- ancestral records.  DECODE: all of them once h_t is back.  FUSED:
  // the parent's own step-(t-1) record as soon as the parent index is back
  // (it needs no ancestry row), together with the parent's row of h_{t-1};
  // then the records of steps <= t-2 once that row is back.
  bool fok[CHAIN];
  fok[NA] = true;
  auto load_record = [&](int j, int slot) {
    const char* ks = k_slab(j);
#pragma unroll
    for (int c = 0; c < C8; ++c) kr[j][c].load(ks, slot * kstride + li * EPL * IOB + c * K8::kBytes);
    abr[j] = load_ab(j, slot);
    vr[j].load(v_slab(j), slot * vstride + voff);
  };
  if constexpr (FUSED && NA > 0) {
    if constexpr (kScalarPar) {
      if (spar) {
        const int sel = lane >> 4;  // this lane's beam within the wave
        fpar = sel == 0 ? spv.x : sel == 1 ? spv.y : sel == 2 ? spv.z : spv.w;
      }
    }
    fpok = unsigned(fpar) < unsigned(p.W_prev);
    const int pf = fpok ? fpar : 0;
    fsrc[NA - 1] = pf;
    fok[NA - 1] = fpok;
    load_record(NA - 1, pf);
    if (tab) {
#pragma unroll
      for (int j = 0; j < NA - 1; ++j) fsrc[j] = anc_lds[pf * (NA - 1) + j];
    } else {
#pragma unroll
      for (int j = 0; j < NA - 1; ++j) fsrc[j] = anc_r[pf * tmax + j];
      // The row is the last load issued, and the records below need it:
      // wait here, inside the branch, so that the join does not make the
      // staged-table path wait for the parent's record as well.
      if constexpr (NA >= 2) __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < NA - 1; ++j) {
      fok[j] = fpok && slot_ok(j, fsrc[j]);
      load_record(j, fok[j] ? fsrc[j] : 0);
    }
  } else {
#pragma unroll
    for (int j = 0; j < NA; ++j) {
      fok[j] = slot_ok(j, fsrc[j]);
      load_record(j, fok[j] ? fsrc[j] : 0);
    }
  }

  // ---- shared-state rows of this wave in MFMA A-fragment order, issued
  // last: they are needed only after the fold and the barrier, and are L2
  // hits for all but the first workgroup of a head on each XCD.  Lane l
  // holds row 16 MB w + 4 MB (m/4) + 4 mb + (m%4) (m = l % 16) and columns
  // 32 ks + 8 (l/16) + [0, 8); the row permutation makes a lane's
  // accumulator rows consecutive state rows.  Step 0 reads fp32 S_ctx and
  // splits it into bf16 hi/lo in registers (tile-0 workgroups store the
  // split fragments in the workspace); later steps read the stored
  // fragments, 1 KiB contiguous per wave-wide load.
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
        const unsigned col = 32 * ks + 8 * (lane >> 4);
        const unsigned off = ((unsigned(unit) * DV + row) * DK + col) * 4u;
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

  // ---- phase 1: fold the query newest -> oldest (scaled form), and sum
  // the value terms g_j v_j of this lane's rows as the g_j appear
  float pt[EPL];
#pragma unroll
  for (int c = 0; c < C8; ++c) qr[c].to_float(pt + 8 * c);
  float vs[VPL];
#pragma unroll
  for (int e = 0; e < VPL; ++e) vs[e] = 0.f;
  float scale = 1.f;
#pragma unroll
  for (int j = NA; j >= 0; --j) {
    float kf[EPL];
#pragma unroll
    for (int c = 0; c < C8; ++c) kr[j][c].to_float(kf + 8 * c);
    float c0 = 0.f, c1 = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; e += 2) {
      c0 = fmaf(kf[e], pt[e], c0);
      c1 = fmaf(kf[e + 1], pt[e + 1], c1);
    }
    const float cdot = group_sum<LPB>(c0 + c1);
    const float alpha = fok[j] ? abr[j].x : 1.f;
    const float beta = fok[j] ? abr[j].y : 0.f;
    const float gt = beta * cdot;
    const float gj = scale * gt;
    float vf[VPL];
    vr[j].to_float(vf);
#pragma unroll
    for (int e = 0; e < VPL; ++e) vs[e] = fmaf(gj, vf[e], vs[e]);
#pragma unroll
    for (int e = 0; e < EPL; ++e) pt[e] = fmaf(-gt, kf[e], pt[e]);
    scale *= alpha;
  }
#pragma unroll
  for (int c = 0; c < C8; ++c) {
    const int k0 = li * EPL + 8 * c;
    float x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = scale * pt[8 * c + e];
    uint4 hi, lo;
    split8(x, hi, lo);
    p_lds[0][fb >> 4][k0 >> 5][(k0 >> 3) & 3][fb & 15] = hi;
    p_lds[1][fb >> 4][k0 >> 5][(k0 >> 3) & 3][fb & 15] = lo;
  }
#pragma unroll
  for (int e = 0; e < VPL; e += 4)
    *reinterpret_cast<float4*>(&v_lds[fb][li * VPL + e]) =
        make_float4(vs[e], vs[e + 1], vs[e + 2], vs[e + 3]);

  // ---- FUSED: index h_t and the step-t record into the context
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
      if (!borrow && hv % p.G == 0) {
        char* ks = k_slab(NA);
#pragma unroll
        for (int c = 0; c < C8; ++c)
          kr[NA][c].store(ks, fbeam * kslot + li * EPL * IOB + c * K8::kBytes);
      }
      if (!borrow && li == 0) ab_slab(NA)[fbeam] = abr[NA];
    }
    if (!borrow && fvalid) vr[NA].store(v_slab(NA), fbeam * vslot + voff);
  }
  __syncthreads();

  // ---- phase 2: O = S_ctx . P on MFMA (three bf16 products per block)
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
  // ---- phase 3 follows each block: add the value terms and store RPL
  // consecutive rows per lane.
  // One beam block after the other: its three accumulator chains (hi*hi and
  // the two cross terms) over the k-steps, then its value terms and stores,
  // so that the first block's outputs stream out while the second block's
  // products run (whole step at the headline 25.2 -> 24.9 us against both
  // blocks' products first).
#pragma unroll
  for (int nb = 0; nb < NBLK; ++nb) {
    f32x4 acc[MB], acx[MB], acy[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
      acx[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
      acy[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    uint4 bh[KS], bl[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      bh[ks] = p_lds[0][nb][ks][g4][lane & 15];
      bl[ks] = p_lds[1][nb][ks][g4][lane & 15];
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        acc[mb] = mfma_bf16(A[ks][mb][0], bh[ks], acc[mb]);
        acx[mb] = mfma_bf16(A[ks][mb][0], bl[ks], acx[mb]);
        acy[mb] = mfma_bf16(A[ks][mb][1], bh[ks], acy[mb]);
      }
    const int bl2 = nb * 16 + (lane & 15);
    const int sb = b0 + bl2;
    float ov[RPL];
#pragma unroll
    for (int e = 0; e < RPL; e += 4) {
      const float4 v4 = *reinterpret_cast<const float4*>(&v_lds[bl2][rloc + e]);
      const f32x4 x = acx[e >> 2] + acy[e >> 2];
      ov[e] = x[0] + acc[e >> 2][0] + v4.x;
      ov[e + 1] = x[1] + acc[e >> 2][1] + v4.y;
      ov[e + 2] = x[2] + acc[e >> 2][2] + v4.z;
      ov[e + 3] = x[3] + acc[e >> 2][3] + v4.w;
    }
    if (sb < W) {
      const unsigned ooff = (((unsigned(r) * W + sb) * p.HV + hv) * DV + row0) * 4u;
#pragma unroll
      for (int i = 0; i < MB; ++i)
        store_out(p.o, ooff + 16u * i, f32x4{ov[4 * i], ov[4 * i + 1], ov[4 * i + 2], ov[4 * i + 3]});
    }
  }
}

template <int DK, int DV, int DVW, bool BF16, bool FUSED, bool BORROW>
hipError_t launch_chain(int chain, const DecodeParams& prm, unsigned blocks, hipStream_t st) {
  constexpr int NBLK = kDecodeBeamBlocks;
  constexpr int threads = decode_threads(DK, DVW);
  switch (chain) {
#define ONELA_CHAIN_CASE(C)                                                                      \
  case C:                                                                                       \
    decode_kernel<DK, DV, DVW, NBLK, C, BF16, FUSED, BORROW><<<blocks, threads, 0, st>>>(prm);  \
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

template <int DK, int DV, int DVW, bool BF16, bool FUSED>
hipError_t launch_storage(int chain, const DecodeParams& prm, unsigned blocks, hipStream_t st) {
  return prm.borrow ? launch_chain<DK, DV, DVW, BF16, FUSED, true>(chain, prm, blocks, st)
                    : launch_chain<DK, DV, DVW, BF16, FUSED, false>(chain, prm, blocks, st);
}

// Supported (d_k, d_v) pairs and the state rows one workgroup covers:
// DVW = min(d_v, 256) rows in 16*MB-row blocks per wave, MB = DVW / d_k, for
// d_k <= 128 (d = 128 launches that would leave most compute units idle use
// 64-row slices); at d_k = 256, 128-row slices of 8 waves with 16 rows each (a
// 256-row workgroup of 16 waves would launch half as many workgroups, each
// streaming twice the shared state, with 128 registers per lane).
template <bool FUSED>
hipError_t launch_mode(const Shape& s, int step, const DecodeParams& prm, unsigned units,
                       hipStream_t st) {
  const int chain = step + 1;
#define ONELA_SHAPE(DK, DV, DVW)                                                          \
  if (s.dk == DK && s.dv == DV) {                                                        \
    const unsigned blocks = units * unsigned(DV / DVW) * unsigned(prm.ntiles);            \
    return s.bf16 ? launch_storage<DK, DV, DVW, true, FUSED>(chain, prm, blocks, st)    \
                  : launch_storage<DK, DV, DVW, false, FUSED>(chain, prm, blocks, st);  \
  }
#define ONELA_SHAPE_BF16(DK, DV, DVW)                                                     \
  if (s.dk == DK && s.dv == DV && s.bf16) {                                              \
    const unsigned blocks = units * unsigned(DV / DVW) * unsigned(prm.ntiles);            \
    return launch_storage<DK, DV, DVW, true, FUSED>(chain, prm, blocks, st);             \
  }
  ONELA_SHAPE(32, 32, 32)
  ONELA_SHAPE(64, 64, 64)
  // d = 128 launches with fewer workgroups than half the compute units (128
  // beams x 16 heads: 64): 64-row slices of 4 waves, twice the workgroups.
  // Both slice widths hold 16 rows per wave, so the split state that step 0
  // stores has the same layout for either.
  if (s.dk == 128 && s.dv == 128 &&
      2u * units * unsigned(prm.ntiles) <= unsigned(s.cus > 0 ? s.cus : 256)) {
    const unsigned blocks = units * 2u * unsigned(prm.ntiles);
    return s.bf16 ? launch_storage<128, 128, 64, true, FUSED>(chain, prm, blocks, st)
                  : launch_storage<128, 128, 64, false, FUSED>(chain, prm, blocks, st);
  }
  ONELA_SHAPE(128, 128, 128)
  ONELA_SHAPE_BF16(128, 256, 256)
  ONELA_SHAPE_BF16(128, 512, 256)
  ONELA_SHAPE_BF16(256, 256, 128)
  ONELA_SHAPE_BF16(256, 512, 128)
#undef ONELA_SHAPE
#undef ONELA_SHAPE_BF16
  return hipErrorInvalidValue;
}

DecodeParams base_params(const Shape& s, int width, const void* q, float* o, const Arena& a,
                         unsigned* units_out) {
  constexpr int BEAMS = 16 * kDecodeBeamBlocks;
  DecodeParams prm = {};
  prm.q = q;
  prm.o = o;
  prm.s0 = a.s0;
  prm.s_frag = reinterpret_cast<uint4*>(a.s_frag);
  prm.ak = a.k;
  prm.av = a.v;
  prm.ab = a.ab;
  prm.borrow = s.borrow ? 1 : 0;
  for (int j = 0; j < kMaxSteps; ++j) {
    prm.bk[j] = a.bk[j];
    prm.bv[j] = a.bv[j];
    prm.balpha[j] = a.balpha[j];
    prm.bbeta[j] = a.bbeta[j];
    prm.bw[j] = a.bw[j];
  }
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


hipError_t launch_decode(const Shape& s, int step, int width, const void* q, float* o,
                         const Arena& a, hipStream_t st) {
  unsigned units;
  DecodeParams prm = base_params(s, width, q, o, a, &units);
  prm.anc_rd = a.anc[step & 1];
  return launch_mode<false>(s, step, prm, units, st);
}

hipError_t launch_fused_step(const Shape& s, int step, int width, int prev_width,
                             const int* parents, const void* k, const void* v,
                             const float* alpha, const float* beta, const void* q, float* o,
                             int* gather_out, const Arena& a, hipStream_t st) {
  unsigned units;
  DecodeParams prm = base_params(s, width, q, o, a, &units);
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
