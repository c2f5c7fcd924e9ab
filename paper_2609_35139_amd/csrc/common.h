// Device-side building blocks shared by the CacheRepair kernels (gfx950).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cr {

typedef __bf16 bf16;
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

constexpr int WAVE = 64;

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
// bf16 round-to-nearest-even (v_cvt_pk_bf16_f32 on gfx950)
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }

// ---------------------------------------------------------------- vectors
// 8 consecutive elements: one 16-byte access for bf16, two for fp32.
template <typename T> struct Vec8;
template <> struct Vec8<bf16> {
  uint4 raw;
  __device__ __forceinline__ void load(const bf16* p) { raw = *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ void store(bf16* p) const { *reinterpret_cast<uint4*>(p) = raw; }
  __device__ __forceinline__ void zero() { raw = make_uint4(0, 0, 0, 0); }
  __device__ __forceinline__ void to_float(float* f) const {
    const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  __device__ __forceinline__ void from_float(const float* f) {
    bf16 b[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) b[i] = (bf16)f[i];
    raw = *reinterpret_cast<const uint4*>(b);
  }
};
template <> struct Vec8<float> {
  uint4 raw[2];
  __device__ __forceinline__ void load(const float* p) {
    raw[0] = reinterpret_cast<const uint4*>(p)[0];
    raw[1] = reinterpret_cast<const uint4*>(p)[1];
  }
  __device__ __forceinline__ void store(float* p) const {
    reinterpret_cast<uint4*>(p)[0] = raw[0];
    reinterpret_cast<uint4*>(p)[1] = raw[1];
  }
  __device__ __forceinline__ void zero() { raw[0] = raw[1] = make_uint4(0, 0, 0, 0); }
  __device__ __forceinline__ void to_float(float* f) const {
    const uint32_t w[8] = {raw[0].x, raw[0].y, raw[0].z, raw[0].w, raw[1].x, raw[1].y, raw[1].z, raw[1].w};
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = __uint_as_float(w[i]);
  }
  __device__ __forceinline__ void from_float(const float* f) {
    raw[0] = make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]), __float_as_uint(f[3]));
    raw[1] = make_uint4(__float_as_uint(f[4]), __float_as_uint(f[5]), __float_as_uint(f[6]), __float_as_uint(f[7]));
  }
};

// ------------------------------------------------------------ MFMA atoms
// 16x16 output tile.  Operand layout (one wavefront of 64 lanes):
//   A: lane l supplies row (l % 16), k = (l / 16) * KPL + [0, KPL)
//   B: lane l supplies col (l % 16), k = (l / 16) * KPL + [0, KPL)
//   C: lane l holds col (l % 16), rows 4 * (l / 16) + [0, 4)
template <typename T> struct Mma16;
template <> struct Mma16<bf16> {
  static constexpr int KPL = 8, KSTEP = 32;
  typedef bf16x8 frag;
  __device__ __forceinline__ static f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mma16<float> {
  static constexpr int KPL = 1, KSTEP = 4;
  typedef float frag;
  __device__ __forceinline__ static f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

// 32x32 output tile.
//   A: lane l supplies row (l % 32), k = (l / 32) * KPL + [0, KPL)
//   B: lane l supplies col (l % 32), k = (l / 32) * KPL + [0, KPL)
//   C: lane l holds col (l % 32), register i holds row (i/4)*8 + (l/32)*4 + i%4
template <typename T> struct Mma32;
template <> struct Mma32<bf16> {
  static constexpr int KPL = 8, KSTEP = 16;
  typedef bf16x8 frag;
  __device__ __forceinline__ static f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mma32<float> {
  static constexpr int KPL = 1, KSTEP = 2;
  typedef float frag;
  __device__ __forceinline__ static f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

template <typename T, typename F>
__device__ __forceinline__ F load_frag(const T* p) { return *reinterpret_cast<const F*>(p); }

// Pack KPL floats into an operand fragment of type T.
__device__ __forceinline__ bf16x8 pack_frag(const float* f, bf16x8*) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (bf16)f[i];
  return r;
}
__device__ __forceinline__ float pack_frag(const float* f, float*) { return f[0]; }

// Sum of the elements of an operand fragment, accumulated in fp32
// (bf16 pairs through v_dot2_f32_bf16 against (1, 1)).
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float frag_sum(bf16x8 v, float acc) {
  const bf16x2 one = {(bf16)1.0f, (bf16)1.0f};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bf16x2 pr = {v[2 * i], v[2 * i + 1]};
    acc = __builtin_amdgcn_fdot2_f32_bf16(pr, one, acc, false);
  }
  return acc;
}
__device__ __forceinline__ float frag_sum(float v, float acc) { return acc + v; }

// ------------------------------------------------- direct global -> LDS
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void glb_void;

// One 16-byte global -> LDS transfer per lane (global_load_lds_dwordx4): a
// wave writes 64 consecutive 16-byte slots starting at `lds_wave_base`
// (wave-uniform), lane l filling slot l.  Completion is tracked by vmcnt.
__device__ __forceinline__ void dma16(const void* gsrc, void* lds_wave_base) {
  __builtin_amdgcn_global_load_lds((glb_void*)gsrc, (lds_void*)lds_wave_base, 16, 0, 0);
}

// Wait until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Tiles staged in LDS as rows of RB bytes (64, 128 or 256) made of 16-byte
// chunks.  Chunk c of row r lives in slot c ^ ((r / (256 / RB)) % (RB / 16)):
// the rows read together by a 16-lane group of a fragment load then start
// in distinct banks.  A wave's 1 KB DMA round fills 1024 / RB whole rows.
template <int RB>
struct Swz {
  static constexpr int CPR = RB / 16;          // chunks per row
  static constexpr int RPW = 1024 / RB;        // rows per wave DMA round
  __device__ __forceinline__ static int slot(int row, int chunk) {
    return chunk ^ ((row / (256 / RB)) % CPR);
  }
  __device__ __forceinline__ static int offset(int row, int chunk) {
    return row * RB + (slot(row, chunk) << 4);
  }
};
__device__ __forceinline__ int swz128(int row) { return (row >> 1) & 7; }

// --------------------------------------------------------- reductions
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}
__device__ __forceinline__ int wave_min(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, WAVE));
  return v;
}
__device__ __forceinline__ int wave_max(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, WAVE));
  return v;
}

// erf from Abramowitz & Stegun, Handbook of Mathematical Functions, formula
// 7.1.26: erf(x) = 1 - (a1 t + ... + a5 t^5) exp(-x^2), t = 1 / (1 + p x),
// x >= 0, odd extension; |error| <= 1.5e-7.
__device__ __forceinline__ float erf_as7126(float x) {
  const float ax = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(0.3275911f, ax, 1.0f));
  float poly = __builtin_fmaf(1.061405429f, t, -1.453152027f);
  poly = __builtin_fmaf(poly, t, 1.421413741f);
  poly = __builtin_fmaf(poly, t, -0.284496736f);
  poly = __builtin_fmaf(poly, t, 0.254829592f) * t;
  const float e = __builtin_amdgcn_exp2f(-(ax * ax) * 1.4426950408889634f);
  return __builtin_copysignf(__builtin_fmaf(-poly, e, 1.0f), x);
}

// GELU(x) = x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2)).
__device__ __forceinline__ float gelu_erf(float x) {
  return 0.5f * x * (1.0f + erf_as7126(x * 0.70710678118654752f));
}

}  // namespace cr
