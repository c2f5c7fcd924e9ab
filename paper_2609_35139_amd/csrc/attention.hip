// Block-causal flash attention of the repair backbone (gfx950 MFMA).
//
// Query row i may attend to key j iff lo(i) <= j < hi(i), where lo is the
// first token of i's request and hi one past the end of i's chunk: this is
// the mask A_ij = 1[c(j) <= c(i)] of the paper's Section 4.1 restricted to
// one request of a packed batch.  The mask is never materialised: each
// workgroup walks only the key tiles inside the union of its rows' intervals
// (tiles wholly after the rows' chunks or before their request are never
// loaded) and applies per-element masking only on tiles that are not fully
// inside every row's interval.
//
// A workgroup owns 128 queries of one head (32 per wave).  Scores are formed
// transposed, S^T = K Q^T, with 32x32 MFMA atoms, so that each lane holds the
// scores of one query: the online-softmax max and sum are register
// reductions plus one exchange with lane ^ 32.  The K rows of each 32-key
// sub-tile are fed to the MFMA in an order (bits 2 and 3 of the row index
// swapped) that makes the score accumulator registers coincide with the B
// operand of the P V product, so probabilities never leave registers.
// V arrives transposed (vt[head][d][token]) from the QKV epilogue and is
// staged in LDS as [d][key], which turns the A operand of O^T = V^T P^T into
// contiguous 16-byte reads.  K/V tiles are double-buffered through LDS.
#include <climits>

#include "launch.h"

namespace cr {

template <typename T, int D>
struct AttnCfg {
  static constexpr int BQ = 128, BKV = 64;
  static constexpr int VEC = 16 / (int)sizeof(T);
  static constexpr int LDK = D + VEC;      // K tile row (elements)
  static constexpr int LDV = BKV + VEC;    // V^T tile row (elements)
  static constexpr int KVEC = BKV * D / VEC / 256;  // 16-byte loads per thread per tile
};

// A-operand row r of a 32-key sub-tile reads key swap_bits23(r).
__device__ __forceinline__ int swap_bits23(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}
// Key (within a 32-key sub-tile) held by score register i of lane half g.
__device__ __forceinline__ int score_key(int g, int i) { return (i >> 3) * 16 + g * 8 + (i & 7); }

template <typename T, int D>
__global__ __launch_bounds__(256) void attention_kernel(const T* __restrict__ Q,
                                                        const T* __restrict__ Kg,
                                                        const T* __restrict__ Vt,
                                                        T* __restrict__ O, int N, int d_b,
                                                        int n_heads, int64_t n_pad,
                                                        const int* __restrict__ lo_arr,
                                                        const int* __restrict__ hi_arr,
                                                        float scale_log2, int n_qtiles) {
  using C = AttnCfg<T, D>;
  using MM = Mma32<T>;
  using frag = typename MM::frag;
  constexpr int KPL = MM::KPL, KSTEP = MM::KSTEP;
  constexpr int QF = D / KSTEP;          // Q fragments per lane
  constexpr int DT = D / 32;             // 32-row tiles of O^T
  __shared__ __align__(16) T Ks[2][C::BKV * C::LDK];
  __shared__ __align__(16) T Vs[2][D * C::LDV];
  __shared__ int red[2][4];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, ql = lane & 31;
  const int head = blockIdx.x % n_heads;
  const int qt = n_qtiles - 1 - blockIdx.x / n_heads;   // latest (longest) tiles first
  const int q = qt * C::BQ + wave * 32 + ql;
  const bool qvalid = q < N;
  const int lo = qvalid ? lo_arr[q] : 0;
  const int hi = qvalid ? hi_arr[q] : 0;

  // key range of the workgroup and mask-free window of this wave
  {
    const int wlo = wave_min(qvalid ? lo : INT_MAX);
    const int whi = wave_max(qvalid ? hi : 0);
    if (lane == 0) { red[0][wave] = wlo; red[1][wave] = whi; }
  }
  const int wmax_lo = wave_max(qvalid ? lo : INT_MIN);
  const int wmin_hi = wave_min(qvalid ? hi : INT_MAX);
  const int mlo = qvalid ? lo : INT_MIN, mhi = qvalid ? hi : INT_MAX;
  __syncthreads();
  const int kv_begin = min(min(red[0][0], red[0][1]), min(red[0][2], red[0][3]));
  const int kv_end = max(max(red[1][0], red[1][1]), max(red[1][2], red[1][3]));
  const int kb = (kv_begin / C::BKV) * C::BKV;
  const int ntiles = (kv_end - kb + C::BKV - 1) / C::BKV;

  // Q^T fragments stay in registers: col = query, k = d
  frag qf[QF];
#pragma unroll
  for (int s = 0; s < QF; ++s) {
    if (qvalid) qf[s] = load_frag<T, frag>(Q + (int64_t)q * d_b + head * D + s * KSTEP + g * KPL);
    else qf[s] = frag{};
  }

  const T* kbase = Kg + head * D;
  const T* vbase = Vt + (int64_t)head * D * n_pad;
  uint4 rk[C::KVEC], rv[C::KVEC];
  auto gload = [&](int k0) {
#pragma unroll
    for (int p = 0; p < C::KVEC; ++p) {
      const int v = tid + p * 256;
      const int kr = v / (D / C::VEC), kc = (v % (D / C::VEC)) * C::VEC;
      const int key = k0 + kr;
      rk[p] = key < N ? *reinterpret_cast<const uint4*>(kbase + (int64_t)key * d_b + kc)
                      : make_uint4(0, 0, 0, 0);
      const int vr = v / (C::BKV / C::VEC), vc = (v % (C::BKV / C::VEC)) * C::VEC;
      rv[p] = *reinterpret_cast<const uint4*>(vbase + (int64_t)vr * n_pad + k0 + vc);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int p = 0; p < C::KVEC; ++p) {
      const int v = tid + p * 256;
      const int kr = v / (D / C::VEC), kc = (v % (D / C::VEC)) * C::VEC;
      *reinterpret_cast<uint4*>(&Ks[buf][kr * C::LDK + kc]) = rk[p];
      const int vr = v / (C::BKV / C::VEC), vc = (v % (C::BKV / C::VEC)) * C::VEC;
      *reinterpret_cast<uint4*>(&Vs[buf][vr * C::LDV + vc]) = rv[p];
    }
  };

  f32x16 oacc[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d) oacc[d] = f32x16{};
  float m = -INFINITY, lsum = 0.f;
  const int krow = swap_bits23(ql);

  if (ntiles > 0) {
    gload(kb);
    lstore(0);
  }
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int cur = t & 1;
    const int k0 = kb + t * C::BKV;
    if (t + 1 < ntiles) gload(k0 + C::BKV);

    // S^T for two 32-key sub-tiles
    f32x16 s[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      s[rt] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < QF; ++ks) {
        const frag a = load_frag<T, frag>(&Ks[cur][(rt * 32 + krow) * C::LDK + ks * KSTEP + g * KPL]);
        s[rt] = MM::mma(a, qf[ks], s[rt]);
      }
    }
    const bool need_mask = !(k0 >= wmax_lo && k0 + C::BKV <= wmin_hi);
    float mx = -INFINITY;
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float v = s[rt][i] * scale_log2;
        if (need_mask) {
          const int key = k0 + rt * 32 + score_key(g, i);
          if (key < mlo || key >= mhi) v = -INFINITY;
        }
        s[rt][i] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32, WAVE));
    const float m_new = fmaxf(m, mx);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = exp2f(m - m_use);
    m = m_new;
    float psum = 0.f;
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = exp2f(s[rt][i] - m_use);
        s[rt][i] = p;
        psum += p;
      }
    lsum = lsum * alpha + psum;
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int i = 0; i < 16; ++i) oacc[d][i] *= alpha;

    // O^T += V^T P^T
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int s2 = 0; s2 < 32 / KSTEP; ++s2) {
        float pv[KPL];
#pragma unroll
        for (int e = 0; e < KPL; ++e) pv[e] = s[rt][s2 * KPL + e];
        const frag b = pack_frag(pv, (frag*)nullptr);
        const int kofs = rt * 32 + score_key(g, s2 * KPL);
#pragma unroll
        for (int d = 0; d < DT; ++d) {
          const frag a = load_frag<T, frag>(&Vs[cur][(d * 32 + ql) * C::LDV + kofs]);
          oacc[d] = MM::mma(a, b, oacc[d]);
        }
      }

    if (t + 1 < ntiles) lstore(cur ^ 1);
    __syncthreads();
  }

  if (!qvalid) return;
  const float total = lsum + __shfl_xor(lsum, 32, WAVE);
  const float inv = 1.0f / total;
  T* orow = O + (int64_t)q * d_b + head * D;
#pragma unroll
  for (int d = 0; d < DT; ++d)
#pragma unroll
    for (int i4 = 0; i4 < 4; ++i4) {
      const int dd = d * 32 + i4 * 8 + g * 4;
      T outv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) outv[e] = from_f32<T>(oacc[d][i4 * 4 + e] * inv);
      if constexpr (sizeof(T) == 2) {
        *reinterpret_cast<uint2*>(orow + dd) = *reinterpret_cast<const uint2*>(outv);
      } else {
        *reinterpret_cast<uint4*>(orow + dd) = *reinterpret_cast<const uint4*>(outv);
      }
    }
}

template <typename T>
hipError_t attention(const T* q, const T* k, const T* vt, T* o, int N, int d_b, int n_heads,
                     int d_head, int64_t n_pad, const int* lo, const int* hi, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  const int n_qtiles = (N + 127) / 128;
  const float scale_log2 = (float)(1.4426950408889634 / __builtin_sqrt((double)d_head));
  dim3 grid(n_qtiles * n_heads);
  if (d_head == 64) {
    hipLaunchKernelGGL((attention_kernel<T, 64>), grid, dim3(256), 0, s, q, k, vt, o, N, d_b,
                       n_heads, n_pad, lo, hi, scale_log2, n_qtiles);
  } else if (d_head == 32) {
    hipLaunchKernelGGL((attention_kernel<T, 32>), grid, dim3(256), 0, s, q, k, vt, o, N, d_b,
                       n_heads, n_pad, lo, hi, scale_log2, n_qtiles);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template hipError_t attention<bf16>(const bf16*, const bf16*, const bf16*, bf16*, int, int, int,
                                    int, int64_t, const int*, const int*, hipStream_t);
template hipError_t attention<float>(const float*, const float*, const float*, float*, int, int,
                                     int, int, int64_t, const int*, const int*, hipStream_t);

}  // namespace cr
