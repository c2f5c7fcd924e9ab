// Tiled MFMA GEMM for the repair network's dense projections (gfx950).
//
// C[M][N] = A[M][K] * B[N][K]^T with both operands K-contiguous (activations
// row-major, weights prepared as [out][in]).  A 256-thread workgroup owns an
// output tile split in four wave quadrants computed with 32x32 MFMA atoms.
// K advances in slabs of 128 bytes per row, fetched straight from global
// memory into an LDS ring with global_load_lds (no register staging); rows
// are XOR-swizzled in LDS so fragment reads are conflict-free.  The fp32 accumulators are then
// staged through LDS so that every epilogue reads and writes whole 16-byte
// row segments (bias, GELU, residual add, RoPE, transposed V, and the
// strided in-place add into the KV cache).
#include "launch.h"

namespace cr {

// Tile geometry: a 2x2 grid of waves, each owning TM x TN MFMA atoms of
// 32x32 (bf16: v_mfma_f32_32x32x16_bf16, fp32: v_mfma_f32_32x32x2_f32; on
// gfx950 the 32x32 atoms sustain several times the rate of the 16x16 ones),
// so the workgroup tile is (64*TM) x (64*TN).  K advances in slabs of one
// 128-byte row per tile row; STAGES slabs live in the LDS ring.
template <typename T, int TM_, int TN_, int STAGES_>
struct GemmTile {
  static constexpr int TM = TM_, TN = TN_, STAGES = STAGES_;
  static constexpr int NW = 4, NT = 256;
  static constexpr int WM = 32 * TM, WN = 32 * TN;
  static constexpr int BM = 2 * WM, BN = 2 * WN;
  static constexpr int BK = 128 / (int)sizeof(T);   // elements per 128-byte row
  static constexpr int VEC = 16 / (int)sizeof(T);   // elements per 16-byte chunk
  static constexpr int A_ROUNDS = BM * 8 / NT;      // 16-byte DMA ops per thread per slab
  static constexpr int B_ROUNDS = BN * 8 / NT;
  static constexpr int OPS = A_ROUNDS + B_ROUNDS;
  static constexpr int STAGE_BYTES = (BM + BN) * 128;
  static constexpr int HC = BN / 2;                 // epilogue handles one column half at a time
  static constexpr int LDC = HC + 4;                // fp32 staging row
  static constexpr size_t LDS_MAIN = (size_t)STAGES * STAGE_BYTES;
  static constexpr size_t LDS_C = (size_t)BM * LDC * sizeof(float);
  static constexpr size_t LDS = LDS_MAIN > LDS_C ? LDS_MAIN : LDS_C;
  static_assert(OPS * (STAGES - 2) <= 63, "vmcnt range");
};

// Epilogues receive a staged block Cs[ROWS][LDC] (fp32) whose element (r, c)
// is output (m0 + r, n0 + c).  Each thread owns one 8-column segment and a
// strided set of rows, so per-column vectors (bias, sigma) are loaded once
// and every global load of the segment's rows is issued before any of them
// is needed.
template <int ROWS, int COLS>
struct SegMap {
  static constexpr int SEG = COLS / 8;            // segments per row
  static constexpr int RSTEP = 256 / SEG;         // rows between a thread's passes
  static constexpr int PASSES = ROWS / RSTEP;
  static_assert(256 % SEG == 0 && ROWS % RSTEP == 0, "segment map");
  __device__ static int col() { return (threadIdx.x % SEG) * 8; }
  __device__ static int row(int p) { return threadIdx.x / SEG + p * RSTEP; }
};

__device__ __forceinline__ void load8f(const float* p, float* v) {
  const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

template <typename T>
struct EpiBias {
  static constexpr bool kFullTile = false;
  T* out; int64_t ldo; const float* bias; const T* resid; int64_t ldr; const T* resid2;
  int64_t ldr2; int gelu;
  template <int ROWS, int COLS, int LDC>
  __device__ void run(const float* Cs, int m0, int n0, int M, int N) const {
    using S = SegMap<ROWS, COLS>;
    const int c = S::col(), gn = n0 + c;
    if (gn >= N) return;
    float b[8];
    load8f(bias + gn, b);
    Vec8<T> rv[S::PASSES], rv2[S::PASSES];
    if (resid) {
#pragma unroll
      for (int p = 0; p < S::PASSES; ++p) {
        const int gm = m0 + S::row(p);
        if (gm < M) rv[p].load(resid + (int64_t)gm * ldr + gn);
      }
    }
    if (resid2) {
#pragma unroll
      for (int p = 0; p < S::PASSES; ++p) {
        const int gm = m0 + S::row(p);
        if (gm < M) rv2[p].load(resid2 + (int64_t)gm * ldr2 + gn);
      }
    }
#pragma unroll
    for (int p = 0; p < S::PASSES; ++p) {
      const int r = S::row(p), gm = m0 + r;
      if (gm >= M) continue;
      float v[8];
      load8f(Cs + r * LDC + c, v);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        v[k] += b[k];
        if (gelu) v[k] = gelu_erf(v[k]);
      }
      if (resid) {
        float rf[8]; rv[p].to_float(rf);
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = rf[k] + v[k];
      }
      if (resid2) {
        float rf[8]; rv2[p].to_float(rf);
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = v[k] + rf[k];
      }
      Vec8<T> o; o.from_float(v); o.store(out + (int64_t)gm * ldo + gn);
    }
  }
};

template <typename T>
struct EpiQKV {
  static constexpr bool kFullTile = false;
  T* q; T* k; T* vt; int64_t n_pad; int d_b, d_head; const float* bias; const int* pos;
  const float2* rope;
  template <int ROWS, int COLS, int LDC>
  __device__ void run(const float* Cs, int m0, int n0, int M, int N) const {
    if (n0 < 2 * d_b) {
      // Q or K: rotate pairs (i, i + d_head/2) of every head by pos * freq_i.
      // The block is head-aligned and never straddles Q/K (d_b % COLS == 0).
      using S = SegMap<ROWS, COLS>;
      T* dst = n0 < d_b ? q : k;
      const int cbase = n0 < d_b ? n0 : n0 - d_b;
      const int half = d_head / 2;
      const int c = S::col(), gn = n0 + c;
      const int hc = c % d_head;
      const bool first = hc < half;
      const int pc = first ? c + half : c - half;
      const int fi = first ? hc : hc - half;
      float bx[8], by[8];
      load8f(bias + gn, bx);
      load8f(bias + n0 + pc, by);
      int pp[S::PASSES];
#pragma unroll
      for (int p = 0; p < S::PASSES; ++p) {
        const int gm = m0 + S::row(p);
        pp[p] = gm < M ? pos[gm] : 0;
      }
#pragma unroll
      for (int p = 0; p < S::PASSES; ++p) {
        const int r = S::row(p), gm = m0 + r;
        if (gm >= M) continue;
        const float4* cs4 = reinterpret_cast<const float4*>(rope + (int64_t)pp[p] * half + fi);
        float x[8], y[8], v[8];
        load8f(Cs + r * LDC + c, x);
        load8f(Cs + r * LDC + pc, y);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float4 t = cs4[e];   // (cos, sin) of pairs 2e and 2e+1
          const float c0 = t.x, s0 = t.y, c1 = t.z, s1 = t.w;
          const float x0 = x[2 * e] + bx[2 * e], y0 = y[2 * e] + by[2 * e];
          const float x1 = x[2 * e + 1] + bx[2 * e + 1], y1 = y[2 * e + 1] + by[2 * e + 1];
          v[2 * e] = first ? x0 * c0 - y0 * s0 : x0 * c0 + y0 * s0;
          v[2 * e + 1] = first ? x1 * c1 - y1 * s1 : x1 * c1 + y1 * s1;
        }
        Vec8<T> o; o.from_float(v); o.store(dst + (int64_t)gm * d_b + cbase + c);
      }
    } else {
      // V: write transposed, vt[head][d][token], 8 tokens per store.  Rows
      // in [M, n_pad) hold values computed from clamped rows: finite padding.
      constexpr int RSEG = ROWS / 8;
      for (int idx = threadIdx.x; idx < COLS * RSEG; idx += 256) {
        const int c = idx / RSEG, r = (idx % RSEG) * 8;
        const int gn = n0 + c, gm = m0 + r;
        if (gn >= N || gm + 8 > n_pad) continue;
        const int vc = gn - 2 * d_b;
        const float bb = bias[gn];
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = Cs[(r + e) * LDC + c] + bb;
        Vec8<T> o; o.from_float(v);
        o.store(vt + (int64_t)vc * n_pad + gm);
      }
    }
  }
};

// Coordinate j = ((l*2 + kv)*H + h)*d_h + i of the residual in the strided
// cache: pointer of token 0's element, and whether it is a K coordinate.
template <typename T>
__device__ __forceinline__ T* kv_coord(T* kv, const KvStrides& ks, int j, bool* is_k) {
  const int i = j % ks.head_dim;
  const int seg = j / ks.head_dim;
  const int h = seg % ks.n_kv_heads;
  const int lk = seg / ks.n_kv_heads;
  *is_k = (lk & 1) == 0;
  return kv + (int64_t)(lk >> 1) * ks.layer + (int64_t)(lk & 1) * ks.kv + (int64_t)h * ks.head + i;
}

template <typename T>
struct EpiExpand {
  static constexpr bool kFullTile = false;
  T* kv; KvStrides ks; const float* bias; const float* sigma; int mode; const int* keep;
  template <int ROWS, int COLS, int LDC>
  __device__ void run(const float* Cs, int m0, int n0, int M, int N) const {
    using S = SegMap<ROWS, COLS>;
    const int c = S::col(), gn = n0 + c;
    if (gn >= N) return;
    // 8 | d_h keeps a segment in one head
    bool is_k;
    T* base = kv_coord(kv, ks, gn, &is_k);
    if (!(mode & (is_k ? EXPAND_K : EXPAND_V))) return;   // component left stale
    const bool res = mode & EXPAND_RESIDUAL;
    float b[8], sg[8];
    load8f(bias + gn, b);
    load8f(sigma + gn, sg);
    Vec8<T> x[S::PASSES];
    int kp[S::PASSES];
#pragma unroll
    for (int p = 0; p < S::PASSES; ++p) {
      const int gm = m0 + S::row(p);
      kp[p] = (gm < M && keep) ? keep[gm] : 0;
      if (gm < M && res) x[p].load(base + (int64_t)gm * ks.token);
    }
#pragma unroll
    for (int p = 0; p < S::PASSES; ++p) {
      const int r = S::row(p), gm = m0 + r;
      if (gm >= M || kp[p]) continue;
      float a[8], f[8];
      load8f(Cs + r * LDC + c, a);
      if (res) x[p].to_float(f);
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] = (res ? f[e] : 0.f) + sg[e] * (a[e] + b[e]);
      x[p].from_float(f);
      x[p].store(base + (int64_t)gm * ks.token);
    }
  }
};

// Output add followed by the target model's rotation of every key head
// (global placement), on a fully staged tile: a thread owns 8 rotate-half
// pairs (columns c .. c+7 and c+half .. c+half+7 of one head) of a set of
// rows, so both members of every pair are rotated in registers.  Requires
// head_dim <= 128 (a head never straddles two 128-column tiles).
template <typename T>
struct EpiExpandRope {
  static constexpr bool kFullTile = true;
  T* kv; KvStrides ks; const float* bias; const float* sigma; int mode; const int* keep;
  const float2* rope;   // [M][head_dim/2] scaled (cos, sin)
  template <int ROWS, int COLS, int LDC>
  __device__ void run(const float* Cs, int m0, int n0, int M, int N) const {
    constexpr int PAIRS = COLS / 16;               // 8-pair groups per tile row
    constexpr int RSTEP = 256 / PAIRS, PASSES = ROWS / RSTEP;
    const int dh = ks.head_dim, half = dh / 2, sph = half / 8;
    const int p = threadIdx.x % PAIRS;
    const int c1 = (p / sph) * dh + (p % sph) * 8, c2 = c1 + half;
    const int g1 = n0 + c1, g2 = n0 + c2;
    if (g2 >= N) return;
    bool is_k;
    T* b1 = kv_coord(kv, ks, g1, &is_k);
    T* b2 = b1 + half;
    const int i0 = g1 % dh;
    const bool on = mode & (is_k ? EXPAND_K : EXPAND_V);
    if (!on && !is_k) return;                      // stale V: nothing to write
    const bool res = mode & EXPAND_RESIDUAL;
    float bb1[8], bb2[8], s1[8], s2[8];
    load8f(bias + g1, bb1); load8f(bias + g2, bb2);
    load8f(sigma + g1, s1); load8f(sigma + g2, s2);
    Vec8<T> x1[PASSES], x2[PASSES];
    int kp[PASSES];
    float4 cs[PASSES][4];
#pragma unroll
    for (int q = 0; q < PASSES; ++q) {
      const int gm = m0 + threadIdx.x / PAIRS + q * RSTEP;
      kp[q] = (gm < M && keep) ? keep[gm] : 0;
      if (gm < M) {
        x1[q].load(b1 + (int64_t)gm * ks.token);
        x2[q].load(b2 + (int64_t)gm * ks.token);
        if (is_k) {
          const float4* t4 = reinterpret_cast<const float4*>(rope + (int64_t)gm * half + i0);
#pragma unroll
          for (int e = 0; e < 4; ++e) cs[q][e] = t4[e];
        }
      }
    }
#pragma unroll
    for (int q = 0; q < PASSES; ++q) {
      const int r = threadIdx.x / PAIRS + q * RSTEP, gm = m0 + r;
      if (gm >= M) continue;
      float y1[8], y2[8];
      x1[q].to_float(y1);
      x2[q].to_float(y2);
      if (on && !kp[q]) {
        float a1[8], a2[8];
        load8f(Cs + r * LDC + c1, a1);
        load8f(Cs + r * LDC + c2, a2);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          y1[e] = (res ? y1[e] : 0.f) + s1[e] * (a1[e] + bb1[e]);
          y2[e] = (res ? y2[e] : 0.f) + s2[e] * (a2[e] + bb2[e]);
        }
      } else if (!is_k) {
        continue;
      }
      if (is_k) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float4 t = cs[q][e];   // (cos, sin) of pairs 2e and 2e+1
          const float u0 = y1[2 * e], v0 = y2[2 * e], u1 = y1[2 * e + 1], v1 = y2[2 * e + 1];
          y1[2 * e] = t.x * u0 - t.y * v0;
          y2[2 * e] = t.x * v0 + t.y * u0;
          y1[2 * e + 1] = t.z * u1 - t.w * v1;
          y2[2 * e + 1] = t.z * v1 + t.w * u1;
        }
      }
      x1[q].from_float(y1);
      x2[q].from_float(y2);
      x1[q].store(b1 + (int64_t)gm * ks.token);
      x2[q].store(b2 + (int64_t)gm * ks.token);
    }
  }
};

// Wait until slab kt of the ring has landed: `ahead` later slabs may still
// be in flight (OPS DMA operations each).
template <int OPS, int MAXA>
__device__ __forceinline__ void wait_slab(int ahead) {
  if constexpr (MAXA >= 3) { if (ahead >= 3) { wait_vmcnt<3 * OPS>(); return; } }
  if constexpr (MAXA >= 2) { if (ahead >= 2) { wait_vmcnt<2 * OPS>(); return; } }
  if constexpr (MAXA >= 1) { if (ahead >= 1) { wait_vmcnt<OPS>(); return; } }
  wait_vmcnt<0>();
}

template <typename T, typename G, typename Epi>
__global__ __launch_bounds__(256) void gemm_nt_kernel(const T* __restrict__ A, int64_t lda,
                                                      const T* __restrict__ B, int64_t ldb,
                                                      int M, int N, int K, Epi epi) {
  using MM = Mma32<T>;
  using frag = typename MM::frag;
  constexpr int LDCF = G::BN + 4;                    // full-tile staging row
  constexpr size_t LDS_FULL = Epi::kFullTile ? (size_t)G::BM * LDCF * sizeof(float) : 0;
  __shared__ __align__(1024) char smem[G::LDS > LDS_FULL ? G::LDS : LDS_FULL];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m0 = blockIdx.y * G::BM, n0 = blockIdx.x * G::BN;
  const int wm = (wave >> 1) * G::WM, wn = (wave & 1) * G::WN;

  // DMA sources: in round r a wave fills 1 KB = rows (r*NW + wave)*8 + [0, 8)
  // of the tile; lane l reads the chunk that lands in slot (l & 7) of its row.
  // Rows past M / N are clamped to the last row: they only feed outputs that
  // the epilogue discards.
  const char* asrc[G::A_ROUNDS];
  const char* bsrc[G::B_ROUNDS];
#pragma unroll
  for (int r = 0; r < G::A_ROUNDS; ++r) {
    const int row = (r * G::NW + wave) * 8 + (lane >> 3);
    const int chunk = (lane & 7) ^ swz128(row);
    asrc[r] = reinterpret_cast<const char*>(A + (int64_t)min(m0 + row, M - 1) * lda) + chunk * 16;
  }
#pragma unroll
  for (int r = 0; r < G::B_ROUNDS; ++r) {
    const int row = (r * G::NW + wave) * 8 + (lane >> 3);
    const int chunk = (lane & 7) ^ swz128(row);
    bsrc[r] = reinterpret_cast<const char*>(B + (int64_t)min(n0 + row, N - 1) * ldb) + chunk * 16;
  }
  auto issue = [&](int kt, int stage) {
    char* base = smem + stage * G::STAGE_BYTES;
#pragma unroll
    for (int r = 0; r < G::A_ROUNDS; ++r) dma16(asrc[r] + kt * 128, base + (r * G::NW + wave) * 1024);
#pragma unroll
    for (int r = 0; r < G::B_ROUNDS; ++r)
      dma16(bsrc[r] + kt * 128, base + G::BM * 128 + (r * G::NW + wave) * 1024);
  };

  f32x16 acc[G::TM][G::TN];
#pragma unroll
  for (int i = 0; i < G::TM; ++i)
#pragma unroll
    for (int j = 0; j < G::TN; ++j) acc[i][j] = f32x16{};

  const int KT = K / G::BK;
#pragma unroll
  for (int st = 0; st < G::STAGES - 1; ++st)
    if (st < KT) issue(st, st);

  // fragment rows: wm + i*32 + (lane & 31); all share swizzle ((lane & 15) >> 1)
  const int fr = lane & 31, fsw = (lane & 15) >> 1;
  for (int kt = 0; kt < KT; ++kt) {
    wait_slab<G::OPS, G::STAGES - 2>(min(G::STAGES - 2, KT - 1 - kt));
    __builtin_amdgcn_s_barrier();
    if (kt + G::STAGES - 1 < KT) issue(kt + G::STAGES - 1, (kt + G::STAGES - 1) % G::STAGES);

    const char* as = smem + (kt % G::STAGES) * G::STAGE_BYTES;
    const char* bs = as + G::BM * 128;
#pragma unroll
    for (int ks = 0; ks < G::BK; ks += MM::KSTEP) {
      const int k = ks + (lane >> 5) * MM::KPL;
      const int cofs = (((k / G::VEC) ^ fsw) << 4) + (k % G::VEC) * (int)sizeof(T);
      frag af[G::TM], bfr[G::TN];
#pragma unroll
      for (int i = 0; i < G::TM; ++i)
        af[i] = *reinterpret_cast<const frag*>(as + (wm + i * 32 + fr) * 128 + cofs);
#pragma unroll
      for (int j = 0; j < G::TN; ++j)
        bfr[j] = *reinterpret_cast<const frag*>(bs + (wn + j * 32 + fr) * 128 + cofs);
#pragma unroll
      for (int i = 0; i < G::TM; ++i)
#pragma unroll
        for (int j = 0; j < G::TN; ++j) acc[i][j] = MM::mma(af[i], bfr[j], acc[i][j]);
    }
  }

  // Epilogue in two column halves: the waves owning half p stage their
  // accumulators (32x32 layout: lane holds column lane%32, register
  // v holds row (v/4)*8 + (lane/32)*4 + v%4), then all threads run the
  // epilogue on that half.
  float* Cs = reinterpret_cast<float*>(smem);
  if constexpr (Epi::kFullTile) {
    // epilogues that pair columns across the two halves see the whole tile
    __syncthreads();  // ring no longer read
#pragma unroll
    for (int i = 0; i < G::TM; ++i)
#pragma unroll
      for (int j = 0; j < G::TN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          Cs[(wm + i * 32 + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3)) * LDCF + wn + j * 32 + fr] =
              acc[i][j][v];
    __syncthreads();
    epi.template run<G::BM, G::BN, LDCF>(Cs, m0, n0, M, N);
    return;
  }
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    __syncthreads();  // ring (or the previous half) no longer read
    if ((wave & 1) == p) {
#pragma unroll
      for (int i = 0; i < G::TM; ++i)
#pragma unroll
        for (int j = 0; j < G::TN; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            Cs[(wm + i * 32 + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3)) * G::LDC + j * 32 + fr] =
                acc[i][j][v];
    }
    __syncthreads();
    epi.template run<G::BM, G::HC, G::LDC>(Cs, m0, n0 + p * G::HC, M, N);
  }
}

template <typename T, typename G, typename Epi>
static hipError_t launch_tiled(const T* A, int64_t lda, const T* B, int64_t ldb, int M, int N,
                               int K, const Epi& epi, hipStream_t s) {
  if (M <= 0 || N <= 0) return hipSuccess;
  dim3 grid((N + G::BN - 1) / G::BN, (M + G::BM - 1) / G::BM);
  CR_LAUNCH((gemm_nt_kernel<T, G, Epi>), grid, dim3(256), 0, s, A, lda, B, ldb, M, N, K,
                     epi);
  return hipGetLastError();
}

// 128x128 tiles.  Grids of more than one workgroup per CU use a two-slab
// ring (64 KB, two workgroups resident per CU hide each other's latency);
// grids that fit in one pass over the 256 CUs use a three-slab ring instead.
template <typename T, typename Epi>
static hipError_t launch(const T* A, int64_t lda, const T* B, int64_t ldb, int M, int N, int K,
                         const Epi& epi, hipStream_t s) {
  const int64_t tiles = (int64_t)((M + 127) / 128) * ((N + 127) / 128);
  if (tiles <= 256) return launch_tiled<T, GemmTile<T, 2, 2, 3>>(A, lda, B, ldb, M, N, K, epi, s);
  return launch_tiled<T, GemmTile<T, 2, 2, 2>>(A, lda, B, ldb, M, N, K, epi, s);
}

template <typename T>
hipError_t gemm_bias(const T* A, int64_t lda, const T* B, int64_t ldb, int M, int N, int K,
                     T* out, int64_t ldo, const float* bias, const T* resid, int64_t ldr,
                     bool gelu, hipStream_t s, const T* resid2, int64_t ldr2) {
  EpiBias<T> e{out, ldo, bias, resid, ldr, resid2, ldr2, gelu ? 1 : 0};
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
                       KvStrides ks, const float* bias, const float* sigma, int mode,
                       const int* keep, const float2* key_rope, hipStream_t s) {
  if (key_rope) {
    if (ks.head_dim > 128) return hipErrorInvalidValue;
    EpiExpandRope<T> e{kv, ks, bias, sigma, mode, keep, key_rope};
    return launch<T>(A, lda, B, K, M, N, K, e, s);
  }
  EpiExpand<T> e{kv, ks, bias, sigma, mode, keep};
  return launch<T>(A, lda, B, K, M, N, K, e, s);
}

#define CR_INST(T)                                                                              \
  template hipError_t gemm_bias<T>(const T*, int64_t, const T*, int64_t, int, int, int, T*,    \
                                   int64_t, const float*, const T*, int64_t, bool, hipStream_t, \
                                   const T*, int64_t);                                          \
  template hipError_t gemm_qkv<T>(const T*, int64_t, const T*, int, int, int, int, T*, T*, T*, \
                                  int64_t, const float*, const int*, const float2*, hipStream_t); \
  template hipError_t gemm_expand<T>(const T*, int64_t, const T*, int, int, int, T*, KvStrides, \
                                     const float*, const float*, int, const int*,               \
                                     const float2*, hipStream_t);
CR_INST(bf16)
CR_INST(float)
#undef CR_INST

}  // namespace cr
