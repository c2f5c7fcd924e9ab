// Tiled MFMA GEMM for the repair network's dense projections (gfx950).
//
// C[M][N] = A[M][K] * B[N][K]^T with both operands K-contiguous (activations
// row-major, weights prepared as [out][in]).  A 256-thread workgroup owns a
// 128x128 output tile; each of its four waves owns a 64x64 quadrant computed
// with 16x16 MFMA atoms (bf16: 16x16x32, fp32: 16x16x4).  K advances in
// 128-byte slabs that are double-buffered through LDS: global loads for slab
// k+1 are in flight while slab k is multiplied.  The fp32 accumulators are
// then staged through LDS so that every epilogue reads and writes whole
// 16-byte row segments (bias, GELU, residual add, RoPE, transposed V, and the
// strided in-place add into the KV cache).
#include "launch.h"

namespace cr {

template <typename T>
struct GemmTile {
  static constexpr int BM = 128, BN = 128;
  static constexpr int BK = 128 / (int)sizeof(T);   // 64 bf16 / 32 fp32
  static constexpr int VEC = 16 / (int)sizeof(T);   // elements per 16-byte load
  static constexpr int LDK = BK + VEC;              // padded LDS row (elements)
  static constexpr int TPR = BK / VEC;              // threads per tile row
  static constexpr int RPP = 256 / TPR;             // rows per load pass
  static constexpr int PASSES = BM / RPP;
  static constexpr int WM = 64, WN = 64;
  static constexpr int TM = WM / 16, TN = WN / 16;
  static constexpr int LDC = BN + 4;                // fp32 staging row
  static constexpr size_t LDS_MAIN = 2ull * (BM + BN) * LDK * sizeof(T);
  static constexpr size_t LDS_C = (size_t)BM * LDC * sizeof(float);
  static constexpr size_t LDS = LDS_MAIN > LDS_C ? LDS_MAIN : LDS_C;
};

// Visit the staged tile in 8-column row segments that fall inside [M) x [N).
template <typename T, typename F>
__device__ __forceinline__ void for_each_row8(int m0, int n0, int M, int N, F&& f) {
  using G = GemmTile<T>;
  constexpr int SEG = G::BN / 8;
  for (int idx = threadIdx.x; idx < G::BM * SEG; idx += 256) {
    const int r = idx / SEG, c = (idx % SEG) * 8;
    const int gm = m0 + r, gn = n0 + c;
    if (gm < M && gn < N) f(r, c, gm, gn);
  }
}

template <typename T>
struct EpiBias {
  T* out; int64_t ldo; const float* bias; const T* resid; int64_t ldr; int gelu;
  __device__ void operator()(const float* Cs, int m0, int n0, int M, int N) const {
    using G = GemmTile<T>;
    for_each_row8<T>(m0, n0, M, N, [&](int r, int c, int gm, int gn) {
      float v[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        v[k] = Cs[r * G::LDC + c + k] + bias[gn + k];
        if (gelu) v[k] = gelu_erf(v[k]);
      }
      if (resid) {
        Vec8<T> rv; rv.load(resid + (int64_t)gm * ldr + gn);
        float rf[8]; rv.to_float(rf);
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = rf[k] + v[k];
      }
      Vec8<T> o; o.from_float(v); o.store(out + (int64_t)gm * ldo + gn);
    });
  }
};

template <typename T>
struct EpiQKV {
  T* q; T* k; T* vt; int64_t n_pad; int d_b, d_head; const float* bias; const int* pos;
  const float2* rope;
  __device__ void operator()(const float* Cs, int m0, int n0, int M, int N) const {
    using G = GemmTile<T>;
    if (n0 < 2 * d_b) {
      // Q or K: rotate pairs (i, i + d_head/2) of every head by pos * freq_i.
      T* dst = n0 < d_b ? q : k;
      const int cbase = n0 < d_b ? n0 : n0 - d_b;
      const int half = d_head / 2;
      for_each_row8<T>(m0, n0, M, N, [&](int r, int c, int gm, int gn) {
        const int hc = c % d_head;  // n0 is a multiple of d_head
        const bool first = hc < half;
        const int pc = first ? c + half : c - half;
        const int fi = first ? hc : hc - half;
        const float2* cs = rope + (int64_t)pos[gm] * half + fi;
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x = Cs[r * G::LDC + c + e] + bias[gn + e];
          const float y = Cs[r * G::LDC + pc + e] + bias[gn - c + pc + e];
          const float2 t = cs[e];
          v[e] = first ? x * t.x - y * t.y : x * t.x + y * t.y;
        }
        Vec8<T> o; o.from_float(v); o.store(dst + (int64_t)gm * d_b + cbase + c);
      });
    } else {
      // V: write transposed, vt[head][d][token], 8 tokens per store.  Rows
      // in [M, n_pad) hold bias-only values, keeping the padding finite.
      constexpr int RSEG = G::BM / 8;
      for (int idx = threadIdx.x; idx < G::BN * RSEG; idx += 256) {
        const int c = idx / RSEG, r = (idx % RSEG) * 8;
        const int gn = n0 + c, gm = m0 + r;
        if (gn >= N || gm + 8 > n_pad) continue;
        const int vc = gn - 2 * d_b;
        const float bb = bias[gn];
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = Cs[(r + e) * G::LDC + c] + bb;
        Vec8<T> o; o.from_float(v);
        o.store(vt + (int64_t)vc * n_pad + gm);
      }
    }
  }
};

template <typename T>
struct EpiExpand {
  T* kv; KvStrides ks; const float* bias; const float* sigma;
  __device__ void operator()(const float* Cs, int m0, int n0, int M, int N) const {
    using G = GemmTile<T>;
    for_each_row8<T>(m0, n0, M, N, [&](int r, int c, int gm, int gn) {
      // coordinate j = ((l*2 + kv)*H + h)*d_h + i
      const int i = gn % ks.head_dim;
      const int seg = gn / ks.head_dim;
      const int h = seg % ks.n_kv_heads;
      const int lk = seg / ks.n_kv_heads;
      T* p = kv + (int64_t)(lk >> 1) * ks.layer + (int64_t)(lk & 1) * ks.kv +
             (int64_t)gm * ks.token + (int64_t)h * ks.head + i;
      Vec8<T> x; x.load(p);
      float f[8]; x.to_float(f);
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] = f[e] + sigma[gn + e] * (Cs[r * G::LDC + c + e] + bias[gn + e]);
      x.from_float(f); x.store(p);
    });
  }
};

template <typename T, typename Epi>
__global__ __launch_bounds__(256) void gemm_nt_kernel(const T* __restrict__ A, int64_t lda,
                                                      const T* __restrict__ B, int64_t ldb,
                                                      int M, int N, int K, Epi epi) {
  using G = GemmTile<T>;
  using MM = Mma16<T>;
  using frag = typename MM::frag;
  __shared__ __align__(16) char smem[G::LDS];
  T* As = reinterpret_cast<T*>(smem);
  T* Bs = As + 2 * G::BM * G::LDK;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m0 = blockIdx.y * G::BM, n0 = blockIdx.x * G::BN;
  const int wm = (wave >> 1) * G::WM, wn = (wave & 1) * G::WN;
  const int lr = tid / G::TPR, lc = (tid % G::TPR) * G::VEC;

  uint4 ra[G::PASSES], rb[G::PASSES];
  auto gload = [&](int k0) {
#pragma unroll
    for (int p = 0; p < G::PASSES; ++p) {
      const int row = lr + p * G::RPP;
      const int gm = m0 + row, gn = n0 + row;
      ra[p] = gm < M ? *reinterpret_cast<const uint4*>(A + (int64_t)gm * lda + k0 + lc)
                     : make_uint4(0, 0, 0, 0);
      rb[p] = gn < N ? *reinterpret_cast<const uint4*>(B + (int64_t)gn * ldb + k0 + lc)
                     : make_uint4(0, 0, 0, 0);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int p = 0; p < G::PASSES; ++p) {
      const int row = lr + p * G::RPP;
      *reinterpret_cast<uint4*>(As + (buf * G::BM + row) * G::LDK + lc) = ra[p];
      *reinterpret_cast<uint4*>(Bs + (buf * G::BN + row) * G::LDK + lc) = rb[p];
    }
  };

  f32x4 acc[G::TM][G::TN];
#pragma unroll
  for (int i = 0; i < G::TM; ++i)
#pragma unroll
    for (int j = 0; j < G::TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int KT = K / G::BK;
  const int fr = lane & 15, fk = (lane >> 4) * MM::KPL;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) gload((kt + 1) * G::BK);
    const T* as = As + cur * G::BM * G::LDK;
    const T* bs = Bs + cur * G::BN * G::LDK;
#pragma unroll
    for (int ks = 0; ks < G::BK; ks += MM::KSTEP) {
      frag af[G::TM], bfr[G::TN];
#pragma unroll
      for (int i = 0; i < G::TM; ++i)
        af[i] = load_frag<T, frag>(as + (wm + i * 16 + fr) * G::LDK + ks + fk);
#pragma unroll
      for (int j = 0; j < G::TN; ++j)
        bfr[j] = load_frag<T, frag>(bs + (wn + j * 16 + fr) * G::LDK + ks + fk);
#pragma unroll
      for (int i = 0; i < G::TM; ++i)
#pragma unroll
        for (int j = 0; j < G::TN; ++j) acc[i][j] = MM::mma(af[i], bfr[j], acc[i][j]);
    }
    if (kt + 1 < KT) lstore(cur ^ 1);
    __syncthreads();
  }

  float* Cs = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int i = 0; i < G::TM; ++i)
#pragma unroll
    for (int j = 0; j < G::TN; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        Cs[(wm + i * 16 + (lane >> 4) * 4 + e) * G::LDC + wn + j * 16 + fr] = acc[i][j][e];
  __syncthreads();
  epi(Cs, m0, n0, M, N);
}

template <typename T, typename Epi>
static hipError_t launch(const T* A, int64_t lda, const T* B, int64_t ldb, int M, int N, int K,
                         const Epi& epi, hipStream_t s) {
  using G = GemmTile<T>;
  if (M <= 0 || N <= 0) return hipSuccess;
  dim3 grid((N + G::BN - 1) / G::BN, (M + G::BM - 1) / G::BM);
  hipLaunchKernelGGL((gemm_nt_kernel<T, Epi>), grid, dim3(256), 0, s, A, lda, B, ldb, M, N, K, epi);
  return hipGetLastError();
}

template <typename T>
hipError_t gemm_bias(const T* A, int64_t lda, const T* B, int64_t ldb, int M, int N, int K,
                     T* out, int64_t ldo, const float* bias, const T* resid, int64_t ldr,
                     bool gelu, hipStream_t s) {
  EpiBias<T> e{out, ldo, bias, resid, ldr, gelu ? 1 : 0};
  return launch<T>(A, lda, B, ldb, M, N, K, e, s);
}

template <typename T>
hipError_t gemm_qkv(const T* A, int64_t lda, const T* B, int M, int K, int d_b, int d_head,
                    T* q, T* k, T* vt, int64_t n_pad, const float* bias, const int* pos,
                    const float2* rope, hipStream_t s) {
  EpiQKV<T> e{q, k, vt, n_pad, d_b, d_head, bias, pos, rope};
  // the grid covers rows up to roundup(M, 128) == n_pad, so the transposed V
  // padding is written too (A rows >= M read as zero)
  return launch<T>(A, lda, B, K, M, 3 * d_b, K, e, s);
}

template <typename T>
hipError_t gemm_expand(const T* A, int64_t lda, const T* B, int M, int N, int K, T* kv,
                       KvStrides ks, const float* bias, const float* sigma, hipStream_t s) {
  EpiExpand<T> e{kv, ks, bias, sigma};
  return launch<T>(A, lda, B, K, M, N, K, e, s);
}

#define CR_INST(T)                                                                              \
  template hipError_t gemm_bias<T>(const T*, int64_t, const T*, int64_t, int, int, int, T*,    \
                                   int64_t, const float*, const T*, int64_t, bool, hipStream_t); \
  template hipError_t gemm_qkv<T>(const T*, int64_t, const T*, int, int, int, int, T*, T*, T*, \
                                  int64_t, const float*, const int*, const float2*, hipStream_t); \
  template hipError_t gemm_expand<T>(const T*, int64_t, const T*, int, int, int, T*, KvStrides, \
                                     const float*, const float*, hipStream_t);
CR_INST(bf16)
CR_INST(float)
#undef CR_INST

}  // namespace cr
