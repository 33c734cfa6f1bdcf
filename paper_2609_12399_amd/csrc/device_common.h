// Device helpers shared by the decode kernels of libonela (gfx950).
#pragma once

#include <hip/hip_runtime.h>

namespace onela {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Pointer to a byte offset from a base (32-bit offsets keep per-lane address
// arithmetic in 32 bits; every region is smaller than 2 GiB).
template <typename T>
__device__ inline T* at(void* base, unsigned off) {
  return reinterpret_cast<T*>(static_cast<char*>(base) + off);
}
template <typename T>
__device__ inline const T* at(const void* base, unsigned off) {
  return reinterpret_cast<const T*>(static_cast<const char*>(base) + off);
}

// N consecutive io elements (bf16 bits or fp32), raw, moved as whole
// vectors of 8, 16 or 32 bytes.
template <bool BF16, int N>
struct RawV {
  static constexpr int kWords = BF16 ? N / 2 : N;
  static constexpr int kBytes = kWords * 4;
  static_assert(kWords == 2 || kWords == 4 || kWords == 8, "8, 16 or 32 bytes");
  unsigned w[kWords];
  __device__ void load(const void* base, unsigned off) {
    if constexpr (kWords == 2) {
      const uint2 u = *at<uint2>(base, off);
      w[0] = u.x; w[1] = u.y;
    } else {
#pragma unroll
      for (int i = 0; i < kWords / 4; ++i) {
        const uint4 u = *at<uint4>(base, off + 16 * i);
        w[4 * i] = u.x; w[4 * i + 1] = u.y; w[4 * i + 2] = u.z; w[4 * i + 3] = u.w;
      }
    }
  }
  __device__ void store(void* base, unsigned off) const {
    if constexpr (kWords == 2) {
      *at<uint2>(base, off) = make_uint2(w[0], w[1]);
    } else {
#pragma unroll
      for (int i = 0; i < kWords / 4; ++i)
        *at<uint4>(base, off + 16 * i) =
            make_uint4(w[4 * i], w[4 * i + 1], w[4 * i + 2], w[4 * i + 3]);
    }
  }
  __device__ void to_float(float* x) const {
#pragma unroll
    for (int i = 0; i < kWords; ++i) {
      if constexpr (BF16) {
        x[2 * i] = __uint_as_float(w[i] << 16);
        x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
      } else {
        x[i] = __uint_as_float(w[i]);
      }
    }
  }
};

// Two floats rounded to bf16 (round to nearest even), a in the low half.  The
// pair is converted as one vector so that it becomes a single two-source
// v_cvt_pk_bf16_f32; converted one by one, each takes its own conversion
// plus a shift and a merge.
__device__ inline unsigned pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(unsigned, __builtin_convertvector(f32x2{a, b}, bf16x2));
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

// Store of 16 output bytes, at byte offset off of base, that the launch never
// reads again: non-temporal and at device scope (nt sc1), so the lines stream
// out to memory during the launch rather than waiting, dirty in the XCD's L2,
// for the write-back at the launch's end.  A buffer store, so that the
// compiler sees it (and its register hazards).  Measured at 16 heads x 512
// beams: plain stores 28.4 us per 4-step decode, non-temporal 26.2,
// non-temporal at device scope 25.5.  Offsets stay below 2^31 (every region
// is smaller than 2 GiB).
__device__ inline void store_out(void* base, unsigned off, f32x4 v) {
  constexpr int kNtSc1 = 2 | 16;  // cache policy bits: nt, sc1
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(base, static_cast<short>(0), 0x7fffffff, 0x00020000);
  __builtin_amdgcn_raw_buffer_store_b128(v, rs, off, 0, kNtSc1);
}

template <int CTRL>
__device__ inline float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x),
                                                               CTRL, 0xF, 0xF, false));
}

// Sum over an aligned group of G consecutive lanes, result in every lane of
// the group.  Within a 16-lane row the exchanges are DPP moves: swap
// neighbours, swap pairs (quad permutes), then mirror within half-rows and
// within the row; wider groups finish with cross-row shuffles.
template <int G>
__device__ inline float group_sum(float x) {
  if constexpr (G >= 2) x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
  if constexpr (G >= 4) x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
  if constexpr (G >= 8) x += dpp<0x141>(x);  // row_half_mirror
  if constexpr (G >= 16) x += dpp<0x140>(x); // row_mirror
  if constexpr (G >= 32) x += __shfl_xor(x, 16);
  if constexpr (G >= 64) x += __shfl_xor(x, 32);
  return x;
}

__device__ inline f32x4 mfma_bf16(const uint4& a, const uint4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

}  // namespace onela
