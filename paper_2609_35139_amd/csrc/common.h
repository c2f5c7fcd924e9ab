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
// Lane l combined with lane l ^ 32 by a commutative operation.
// v_permlane32_swap exchanges the two 32-lane halves of a pair of registers
// without an LDS round trip; given x twice it leaves the lower half's value
// in one result and the upper half's in the other on every lane, so both
// lanes of a pair compute op(lower, upper) and agree bit for bit.  Both
// lanes of a pair must be active.
__device__ __forceinline__ float2 wave_halves(float x) {
  const auto v = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return make_float2(__uint_as_float(v[0]), __uint_as_float(v[1]));
}
__device__ __forceinline__ float halves_sum(float x) {
  const float2 h = wave_halves(x);
  return h.x + h.y;
}
__device__ __forceinline__ float halves_max(float x) {
  const float2 h = wave_halves(x);
  return fmaxf(h.x, h.y);
}
__device__ __forceinline__ int halves_or(int x) {
  const auto v = __builtin_amdgcn_permlane32_swap((unsigned)x, (unsigned)x, false, false);
  return (int)(v[0] | v[1]);
}
// Sum over the wave, the same value on every lane, by register exchanges
// only: within each 16-lane row, DPP partners at lane ^ 1 and lane ^ 2
// (quad permutes), then the mirror images within 8 and within 16 lanes
// (each step pairs groups that already hold equal partial sums); then the
// rows in pairs (v_permlane16_swap) and the halves (v_permlane32_swap).
// All 64 lanes must be active.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_mov<0xB1>(v);    // quad_perm(1, 0, 3, 2): lane ^ 1
  v += dpp_mov<0x4E>(v);    // quad_perm(2, 3, 0, 1): lane ^ 2
  v += dpp_mov<0x141>(v);   // row_half_mirror: lane 7 - i within 8
  v += dpp_mov<0x140>(v);   // row_mirror: lane 15 - i within 16
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  return halves_sum(v);
}

// GELU(x) = x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2)), with erf(z) taken as
// an odd polynomial z * P(z^2) of degree 17 on |z| <= 3.05 and z clamped to
// that interval, the result clamped to [-1, 1].  P's coefficients are a
// weighted least-squares fit to erf, reweighted towards the largest errors
// until they level out (Lawson's iteration), rounded to fp32.  Evaluated in
// fp32 with fused multiply-adds: |GELU error| <= 5.6e-5 for |x| <= 60 and
// <= 1.4e-5 |x| everywhere, far below one bf16 rounding of the result.  No
// transcendental instruction: GELU is the bulk of the FFN's first
// projection epilogue, which is bound by VALU issue.
constexpr float kGeluZ0 = 3.05f;
constexpr float kGeluErfPoly[9] = {1.12824547290802f,      -0.37517496943473816f,
                                   0.11083579063415527f,   -0.024915285408496857f,
                                   0.004159698728471994f,  -0.0004938565543852746f,
                                   3.885807018377818e-05f, -1.795992830011528e-06f,
                                   3.662422187744596e-08f};
__device__ __forceinline__ float gelu_erf(float x) {
  const float z = __builtin_fminf(__builtin_fmaxf(x * 0.70710678118654752f, -kGeluZ0), kGeluZ0);
  const float s = z * z;
  float p = kGeluErfPoly[8];
#pragma unroll
  for (int k = 7; k >= 0; --k) p = __builtin_fmaf(p, s, kGeluErfPoly[k]);
  const float e = __builtin_fminf(__builtin_fmaxf(z * p, -1.0f), 1.0f);
  const float hx = 0.5f * x;
  return __builtin_fmaf(hx, e, hx);
}

}  // namespace cr
