// Tiled MFMA GEMM for the repair network's dense projections (gfx950).
//
// C[M][N] = A[M][K] * B[N][K]^T with both operands K-contiguous (activations
// row-major, weights prepared as [out][in]).  A workgroup owns an output
// tile (128x128 on four waves or 256x256 on eight) split in wave sub-tiles
// computed with 32x32 MFMA atoms.
// K advances in slabs of 128 bytes per row, fetched straight from global
// memory into an LDS ring with global_load_lds (no register staging); rows
// are XOR-swizzled in LDS so fragment reads are conflict-free.  The MFMA
// takes the weight tile as its first operand, so each lane ends with four
// consecutive output columns of one output row: the fp32 tile is staged
// through LDS with 16-byte writes in one pass, after the epilogue has issued
// its own global loads (bias, residuals, the stale cache), and every
// epilogue then reads and writes whole 16-byte row segments (bias, GELU,
// residual adds, RoPE, transposed V, the strided output add into the KV
// cache with optional global placement of the keys).
#include "launch.h"

namespace cr {

// Tile geometry: a WGM x WGN grid of waves, each owning TM x TN MFMA atoms
// of 32x32 (bf16: v_mfma_f32_32x32x16_bf16, fp32: v_mfma_f32_32x32x2_f32),
// so the workgroup tile is (WGM*32*TM) x (WGN*32*TN).  K advances in slabs
// of one 128-byte row per tile row; STAGES slabs live in the LDS ring.  The
// fp32 output tile is staged through LDS over the ring, EPI_ROWS rows at a
// time (the whole tile, or half of it for 256-row tiles).
template <typename T, int TM_, int TN_, int STAGES_, int WGM_ = 2, int WGN_ = 2,
          bool EARLY2_ = false, int KS_ = 1>
struct GemmTile {
  static constexpr int TM = TM_, TN = TN_, STAGES = STAGES_, WGM = WGM_, WGN = WGN_;
  // KS wave groups of WGM x WGN waves each take 1/KS of every slab's k-steps
  // over the whole tile; their fp32 partial tiles are summed in a fixed
  // order through LDS before the epilogue
  static constexpr int KS = KS_;
  // two staging passes: the first pass's epilogue loads go out before the
  // main loop too
  static constexpr bool EARLY2 = EARLY2_;
  static constexpr int NW = WGM * WGN * KS, NT = 64 * NW;
  static constexpr int WM = 32 * TM, WN = 32 * TN;
  static constexpr int BM = WGM * WM, BN = WGN * WN;
  static constexpr int BK = 128 / (int)sizeof(T);   // elements per 128-byte row
  static constexpr int VEC = 16 / (int)sizeof(T);   // elements per 16-byte chunk
  static constexpr int A_ROUNDS = BM * 8 / NT;      // 16-byte DMA ops per thread per slab
  static constexpr int B_ROUNDS = BN * 8 / NT;
  static constexpr int OPS = A_ROUNDS + B_ROUNDS;
  static constexpr int STAGE_BYTES = (BM + BN) * 128;
  static constexpr int LDC = BN + 4;                // fp32 staging row (16-byte aligned rows)
  static constexpr int EPI_ROWS = BM > 128 ? BM / 2 : BM;
  // a single staging pass issues its epilogue loads before the main loop
  static constexpr bool EARLY = EPI_ROWS == BM;
  static constexpr size_t LDS_MAIN = (size_t)STAGES * STAGE_BYTES;
  static constexpr size_t LDS_C = (size_t)EPI_ROWS * LDC * sizeof(float);
  static constexpr size_t LDS = LDS_MAIN > LDS_C ? LDS_MAIN : LDS_C;
  static_assert(OPS * (STAGES - 2) <= 63, "vmcnt range");
  static_assert(A_ROUNDS * NT == BM * 8 && B_ROUNDS * NT == BN * 8, "DMA rounds");
  static_assert(WM % EPI_ROWS == 0 || EPI_ROWS % WM == 0, "staging passes");
  static_assert(KS == 1 || EPI_ROWS == BM, "split-K tiles stage in one pass");
};

// Epilogues see the staged tile Cs[ROWS][LDC] (fp32) whose element (r, c)
// is output (m0 + r, n0 + c).  Each thread owns one 8-column segment and a
// strided set of rows, so per-column vectors (bias, sigma) are loaded once.
// An epilogue has two phases: prefetch() issues its global loads into a
// Pre record before the tile is staged, run() consumes the staged tile.
template <int ROWS, int COLS, int NT>
struct SegMap {
  static constexpr int SEG = COLS / 8;            // segments per row
  static constexpr int RSTEP = NT / SEG;          // rows between a thread's passes
  static constexpr int PASSES = ROWS / RSTEP;
  static_assert(NT % SEG == 0 && ROWS % RSTEP == 0, "segment map");
  __device__ static int col() { return (threadIdx.x % SEG) * 8; }
  __device__ static int row(int p) { return threadIdx.x / SEG + p * RSTEP; }
};

__device__ __forceinline__ void load8f(const float* p, float* v) {
  const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

template <typename T>
struct EpiBias {
  __device__ int b_row(int n) const { return n; }   // output column -> weight row
  static constexpr bool kWide = true;
  // 64-column tiles are fine for bias epilogues (8-column segments)
  static constexpr bool kNarrow = true;
  T* out; int64_t ldo; const float* bias; const T* resid; int64_t ldr; const T* resid2;
  int64_t ldr2; int gelu;
  template <int ROWS, int COLS, int NT>
  struct Pre {
    float b[8];
    Vec8<T> rv[SegMap<ROWS, COLS, NT>::PASSES], rv2[SegMap<ROWS, COLS, NT>::PASSES];
  };
  template <int ROWS, int COLS, int NT>
  __device__ void prefetch(Pre<ROWS, COLS, NT>& p, int m0, int n0, int M, int N) const {
    using S = SegMap<ROWS, COLS, NT>;
    const int gn = n0 + S::col();
    if (gn >= N) return;
    load8f(bias + gn, p.b);
#pragma unroll
    for (int q = 0; q < S::PASSES; ++q) {
      const int gm = m0 + S::row(q);
      if (gm >= M) continue;
      if (resid) p.rv[q].load(resid + (int64_t)gm * ldr + gn);
      if (resid2) p.rv2[q].load(resid2 + (int64_t)gm * ldr2 + gn);
    }
  }
  template <int ROWS, int COLS, int LDC, int NT>
  __device__ void run(const float* Cs, const Pre<ROWS, COLS, NT>& p, int m0, int n0, int M,
                      int N) const {
    using S = SegMap<ROWS, COLS, NT>;
    const int c = S::col(), gn = n0 + c;
    if (gn >= N) return;
    // without GELU the rows run as straight-line code (-18% for a 256x256
    // bias epilogue); with it, element by element as written (faster than
    // the straight-line form, which holds more values in flight)
    if (!gelu) {
      rows<ROWS, COLS, LDC, NT, false>(Cs, p, m0, M, c, gn);
      return;
    }
    rows<ROWS, COLS, LDC, NT, true>(Cs, p, m0, M, c, gn);
  }
  template <int ROWS, int COLS, int LDC, int NT, bool G>
  __device__ void rows(const float* Cs, const Pre<ROWS, COLS, NT>& p, int m0, int M, int c,
                       int gn) const {
    using S = SegMap<ROWS, COLS, NT>;
#pragma unroll
    for (int q = 0; q < S::PASSES; ++q) {
      const int r = S::row(q), gm = m0 + r;
      if (gm >= M) continue;
      float v[8];
      load8f(Cs + r * LDC + c, v);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        v[k] += p.b[k];
        if (G && gelu) v[k] = gelu_erf(v[k]);
      }
      if (resid) {
        float rf[8]; p.rv[q].to_float(rf);
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = rf[k] + v[k];
      }
      if (resid2) {
        float rf[8]; p.rv2[q].to_float(rf);
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = v[k] + rf[k];
      }
      Vec8<T> o; o.from_float(v); o.store(out + (int64_t)gm * ldo + gn);
    }
  }
};

// QKV projection in the weights' own column order [Q | K | V] on 128-column
// tiles (each inside Q, K or V and head-aligned, d_b % 128 == 0).
template <typename T>
struct EpiQKV {
  static constexpr bool kWide = false;   // head-aligned 128-column tiles
  static constexpr bool kNarrow = false;
  __device__ int b_row(int n) const { return n; }   // output column -> weight row
  T* q; T* k; T* vt; int64_t n_pad; int d_b, d_head; const float* bias;
  const float2* rope;   // (cos, sin) per token
  template <int ROWS, int COLS, int NT>
  struct Pre { float bx[8], by[8]; };
  template <int ROWS, int COLS, int NT>
  __device__ void prefetch(Pre<ROWS, COLS, NT>& p, int m0, int n0, int M, int N) const {
    if (n0 >= 2 * d_b) return;      // V tiles load their bias per column in run()
    using S = SegMap<ROWS, COLS, NT>;
    const int half = d_head / 2;
    const int c = S::col(), hc = c % d_head;
    const int pc = hc < half ? c + half : c - half;
    load8f(bias + n0 + c, p.bx);
    load8f(bias + n0 + pc, p.by);
  }
  template <int ROWS, int COLS, int LDC, int NT>
  __device__ void run(const float* Cs, const Pre<ROWS, COLS, NT>& p, int m0, int n0, int M,
                      int N) const {
    if (n0 < 2 * d_b) {
      // Q or K: rotate pairs (i, i + d_head/2) of every head by pos * freq_i.
      // The tile is head-aligned and never straddles Q/K (d_b % COLS == 0).
      // Q leaves scaled by log2(e)/sqrt(d_head) (the attention works in exp2
      // units); K rows in [M, n_pad) get finite values from clamped rows
      // (padding read by the attention's last key tile).
      using S = SegMap<ROWS, COLS, NT>;
      const bool is_q = n0 < d_b;
      T* dst = is_q ? q : k;
      const int rows_out = is_q ? M : (int)n_pad;
      const float osc = is_q ? 1.4426950408889634f / __builtin_sqrtf((float)d_head) : 1.0f;
      const int cbase = n0 < d_b ? n0 : n0 - d_b;
      const int half = d_head / 2;
      const int c = S::col();
      const int hc = c % d_head;
      const bool first = hc < half;
      const int pc = first ? c + half : c - half;
      const int fi = first ? hc : hc - half;
      // the (cos, sin) rows of a group of passes are loaded together
      // (fewer beside the 256x256 tile, whose other half still holds its
      // accumulators)
      constexpr int GRP = S::PASSES >= 4 && NT == 256 ? 4 : (S::PASSES >= 2 ? 2 : 1);
#pragma unroll
      for (int q0 = 0; q0 < S::PASSES; q0 += GRP) {
      float4 cs[GRP][4];
#pragma unroll
      for (int q = 0; q < GRP; ++q) {
        // rows past M (K padding) take token 0's rotation: finite, never used
        const int gm = m0 + S::row(q0 + q);
        const float4* t4 =
            reinterpret_cast<const float4*>(rope + (int64_t)(gm < M ? gm : 0) * half + fi);
#pragma unroll
        for (int e = 0; e < 4; ++e) cs[q][e] = t4[e];
      }
#pragma unroll
      for (int q = 0; q < GRP; ++q) {
        const int qq = q0 + q;
        const int r = S::row(qq), gm = m0 + r;
        if (gm >= rows_out) continue;
        float x[8], y[8], v[8];
        load8f(Cs + r * LDC + c, x);
        load8f(Cs + r * LDC + pc, y);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float4 t = cs[q][e];   // (cos, sin) of pairs 2e and 2e+1
          const float x0 = x[2 * e] + p.bx[2 * e], y0 = y[2 * e] + p.by[2 * e];
          const float x1 = x[2 * e + 1] + p.bx[2 * e + 1], y1 = y[2 * e + 1] + p.by[2 * e + 1];
          v[2 * e] = (first ? x0 * t.x - y0 * t.y : x0 * t.x + y0 * t.y) * osc;
          v[2 * e + 1] = (first ? x1 * t.z - y1 * t.w : x1 * t.z + y1 * t.w) * osc;
        }
        Vec8<T> o; o.from_float(v); o.store(dst + (int64_t)gm * d_b + cbase + c);
      }
      }
    } else {
      // V: written transposed, vt[head][d][token], 8 tokens per 16-byte
      // store.  Consecutive threads take consecutive columns, so the column
      // reads of the staged tile are conflict-free.  Rows in [M, n_pad) hold
      // values computed from clamped rows: finite padding.
      constexpr int RSEG = ROWS / 8;
      for (int idx = threadIdx.x; idx < COLS * RSEG; idx += NT) {
        const int c = idx % COLS, r = (idx / COLS) * 8;
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

// QKV projection with the output columns taken head by head: tile column
// n is weight row b_row(n), so that columns [3*d_head*h, 3*d_head*(h+1))
// hold Q, K and V of head h.  A 192-column tile then holds whole heads
// (d_head 32 or 64) and a 256x192 tiling of the headline shape is exactly
// one tile per CU.  Q and K get the backbone's RoPE (Q also the scale into
// exp2 units) and are written row-major; V is written transposed.  K rows
// and V^T columns in [M, n_pad) get finite values from clamped A rows.
template <typename T>
struct EpiQKVh {
  static constexpr bool kWide = true;
  static constexpr bool kNarrow = false;
  T* q; T* k; T* vt; int64_t n_pad; int d_b, d_head; const float* bias;
  const float2* rope;   // (cos, sin) per token
  __device__ int b_row(int n) const {
    const int g3 = 3 * d_head, rem = n % g3;
    return (rem / d_head) * d_b + (n / g3) * d_head + rem % d_head;
  }
  // A 192-column tile holds 192 / (3 d_head) heads, so whatever d_head (32 or
  // 64) it has 16 eight-column segments of Q and K and 64 columns of V: every
  // thread's items are known at compile time.  A thread keeps one Q/K segment
  // (threadIdx % QK_SEGS) over rows threadIdx / QK_SEGS + j * NT / QK_SEGS,
  // and one V column over groups of 8 rows.
  template <int ROWS, int COLS, int NT>
  struct Map {
    static_assert(COLS == 192, "head-interleaved 192-column tiles");
    static constexpr int QK_SEGS = COLS / 12;                 // 8-column Q and K segments per row
    static constexpr int QK_ITEMS = ROWS * QK_SEGS / NT;      // per thread
    static constexpr int V_COLS = COLS / 3;
    static constexpr int V_ITEMS = V_COLS * (ROWS / 8) / NT;
    static_assert(NT % QK_SEGS == 0 && QK_ITEMS * NT == ROWS * QK_SEGS, "Q/K items");
    static_assert(NT % V_COLS == 0 && V_ITEMS * NT == V_COLS * (ROWS / 8), "V items");
  };
  struct Seg {
    int c, hh, i, pi, fi, part;
    bool first, col_ok;
  };
  template <int QK_SEGS>
  __device__ Seg seg(int n0, int N) const {
    const int g3 = 3 * d_head, half = d_head / 2;
    const int sg = threadIdx.x % QK_SEGS;
    const int grp = sg / (2 * d_head / 8), w = (sg % (2 * d_head / 8)) * 8;  // w in [0, 2 d_head)
    Seg g;
    g.part = w / d_head;
    g.i = w % d_head;
    g.c = grp * g3 + w;                                   // tile column
    g.hh = (n0 + g.c) / g3;
    g.first = g.i < half;
    g.pi = g.first ? g.i + half : g.i - half;             // partner index in the head
    g.fi = g.first ? g.i : g.i - half;
    g.col_ok = n0 + g.c < N;
    return g;
  }
  // The pass's (cos, sin) entries and biases are loaded before the pass's
  // tile is staged, so their latency hides behind the staging.
  template <int ROWS, int COLS, int NT>
  struct Pre {
    float bx[8], by[8], bb;
    float4 t4[Map<ROWS, COLS, NT>::QK_ITEMS][4];
  };
  // the thread's V column: tile column, head, index in the head
  template <int V_COLS>
  __device__ void vcol(int n0, int& col, int& vh, int& vi) const {
    const int g3 = 3 * d_head, vc = threadIdx.x % V_COLS;
    vi = vc % d_head;
    col = (vc / d_head) * g3 + 2 * d_head + vi;
    vh = (n0 + col) / g3;
  }
  template <int ROWS, int COLS, int NT>
  __device__ void prefetch(Pre<ROWS, COLS, NT>& pr, int m0, int n0, int M, int N) const {
    using MP = Map<ROWS, COLS, NT>;
    const Seg g = seg<MP::QK_SEGS>(n0, N);
    const int half = d_head / 2;
    const int bcol = g.part * d_b + g.hh * d_head;
    if (g.col_ok) { load8f(bias + bcol + g.i, pr.bx); load8f(bias + bcol + g.pi, pr.by); }
#pragma unroll
    for (int j = 0; j < MP::QK_ITEMS; ++j) {
      // rows past M (K padding) take token 0's rotation: finite, never used
      const int gm = m0 + threadIdx.x / MP::QK_SEGS + j * (NT / MP::QK_SEGS);
      const float4* src =
          reinterpret_cast<const float4*>(rope + (int64_t)(gm < M ? gm : 0) * half + g.fi);
#pragma unroll
      for (int e = 0; e < 4; ++e) pr.t4[j][e] = src[e];
    }
    int col, vh, vi;
    vcol<MP::V_COLS>(n0, col, vh, vi);
    if (n0 + col < N) pr.bb = bias[2 * d_b + vh * d_head + vi];
  }
  template <int ROWS, int COLS, int LDC, int NT>
  __device__ void run(const float* Cs, const Pre<ROWS, COLS, NT>& pr, int m0, int n0, int M,
                      int N) const {
    using MP = Map<ROWS, COLS, NT>;
    constexpr int QK_SEGS = MP::QK_SEGS, QK_ITEMS = MP::QK_ITEMS;
    constexpr int V_COLS = MP::V_COLS, V_ITEMS = MP::V_ITEMS;
    const int g3 = 3 * d_head;
    const float qsc = 1.4426950408889634f / __builtin_sqrtf((float)d_head);
    const Seg g = seg<QK_SEGS>(n0, N);
    const int c = g.c, hh = g.hh, i = g.i, pi = g.pi;
    const bool is_q = g.part == 0, first = g.first, col_ok = g.col_ok;
    const int row_end = is_q ? M : (int)n_pad;
    const float* bx = pr.bx;
    const float* by = pr.by;
    const float osc = is_q ? qsc : 1.0f;
#pragma unroll
    for (int j = 0; j < QK_ITEMS; ++j) {
      const int r = threadIdx.x / QK_SEGS + j * (NT / QK_SEGS);
      const int gm = m0 + r;
      if (gm >= row_end || !col_ok) continue;
      float x[8], y[8];
      load8f(Cs + r * LDC + c, x);
      load8f(Cs + r * LDC + c - i + pi, y);
      float v[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float4 t = pr.t4[j][e];   // (cos, sin) of pairs 2e and 2e+1
        const float x0 = x[2 * e] + bx[2 * e], y0 = y[2 * e] + by[2 * e];
        const float x1 = x[2 * e + 1] + bx[2 * e + 1], y1 = y[2 * e + 1] + by[2 * e + 1];
        v[2 * e] = (first ? x0 * t.x - y0 * t.y : x0 * t.x + y0 * t.y) * osc;
        v[2 * e + 1] = (first ? x1 * t.z - y1 * t.w : x1 * t.z + y1 * t.w) * osc;
      }
      Vec8<T> o; o.from_float(v);
      o.store((is_q ? q : k) + (int64_t)gm * d_b + hh * d_head + i);
    }
    // V: transposed, vt[head][d][token], 8 tokens per 16-byte store; a thread
    // keeps one column (consecutive threads take consecutive columns, so the
    // LDS reads are conflict-free)
    int vcl, vh, vi;
    vcol<V_COLS>(n0, vcl, vh, vi);
    if (n0 + vcl >= N) return;
    const float bb = pr.bb;
#pragma unroll
    for (int j = 0; j < V_ITEMS; ++j) {
      const int r = (threadIdx.x / V_COLS + j * (NT / V_COLS)) * 8, gm = m0 + r;
      if (gm + 8 > n_pad) continue;
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = Cs[(r + e) * LDC + vcl] + bb;
      Vec8<T> o; o.from_float(v);
      o.store(vt + (int64_t)(vh * d_head + vi) * n_pad + gm);
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
  __device__ int b_row(int n) const { return n; }   // output column -> weight row
  static constexpr bool kWide = false;
  static constexpr bool kNarrow = false;
  T* kv; KvStrides ks; const float* bias; const float* sigma; int mode; const int* keep;
  T* kvo; KvStrides kso;   // destination when repairing out of place (kvo null: in place)
  // What the prefetch holds: the stale values of the thread's rows and a
  // bitmask of its kept rows; bias and sigma (two 8-float column vectors)
  // are loaded in run() beside a 256x256 tile, whose main loop leaves no
  // registers for them, and prefetched otherwise.
  template <int ROWS, int COLS, int NT>
  struct Pre {
    static constexpr bool kVec = NT == 256;
    float b[kVec ? 8 : 1], sg[kVec ? 8 : 1];
    Vec8<T> x[SegMap<ROWS, COLS, NT>::PASSES];
    unsigned kbits;
  };
  // 8 | d_h keeps a segment in one head
  __device__ bool selected(int gn, T** base) const {
    bool is_k;
    *base = kv_coord(kv, ks, gn, &is_k);
    return mode & (is_k ? EXPAND_K : EXPAND_V);
  }
  template <int ROWS, int COLS, int NT>
  __device__ void prefetch(Pre<ROWS, COLS, NT>& p, int m0, int n0, int M, int N) const {
    using S = SegMap<ROWS, COLS, NT>;
    static_assert(S::PASSES <= 32, "keep bitmask");
    const int gn = n0 + S::col();
    p.kbits = 0;
    if (gn >= N) return;
    T* base;
    const bool sel = selected(gn, &base);
    if (!sel && !kvo) return;                      // unselected component: left stale in place
    if constexpr (Pre<ROWS, COLS, NT>::kVec) {
      if (sel) {
        load8f(bias + gn, p.b);
        load8f(sigma + gn, p.sg);
      }
    }
    const bool need_x = kvo || (mode & EXPAND_RESIDUAL);
#pragma unroll
    for (int q = 0; q < S::PASSES; ++q) {
      const int gm = m0 + S::row(q);
      if (gm < M && keep && keep[gm]) p.kbits |= 1u << q;
      if (gm < M && need_x) p.x[q].load(base + ks.tok(gm));
    }
  }
  template <int ROWS, int COLS, int LDC, int NT>
  __device__ void run(const float* Cs, Pre<ROWS, COLS, NT>& p, int m0, int n0, int M, int N) const {
    using S = SegMap<ROWS, COLS, NT>;
    const int c = S::col(), gn = n0 + c;
    if (gn >= N) return;
    T* base;
    const bool sel = selected(gn, &base);
    if (!sel && !kvo) return;
    bool dummy;
    T* obase = kvo ? kv_coord(kvo, kso, gn, &dummy) : base;
    const bool res = mode & EXPAND_RESIDUAL;
    float bv[8], sv[8];
    if constexpr (Pre<ROWS, COLS, NT>::kVec) {
#pragma unroll
      for (int e = 0; e < 8; ++e) { bv[e] = p.b[e]; sv[e] = p.sg[e]; }
    } else if (sel) {
      load8f(bias + gn, bv);
      load8f(sigma + gn, sv);
    }
#pragma unroll
    for (int q = 0; q < S::PASSES; ++q) {
      const int r = S::row(q), gm = m0 + r;
      if (gm >= M) continue;
      // (no reference that selects between the two stride sets: it would pin
      // the epilogue's arguments to scratch memory)
      const int64_t to = kvo ? kso.tok(gm) : ks.tok(gm);
      if (!sel || (p.kbits >> q & 1u)) {           // stale values: copied when out of place
        if (kvo) p.x[q].store(obase + to);
        continue;
      }
      float a[8], f[8];
      load8f(Cs + r * LDC + c, a);
      if (res) p.x[q].to_float(f);
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] = (res ? f[e] : 0.f) + sv[e] * (a[e] + bv[e]);
      p.x[q].from_float(f);
      p.x[q].store(obase + to);
    }
  }
};

// Output add followed by the target model's rotation of every key head
// (global placement): a thread owns 8 rotate-half pairs (columns c .. c+7 and
// c+half .. c+half+7 of one head) of a set of rows, so both members of every
// pair are rotated in registers.  Requires head_dim <= 128 (a head never
// straddles two 128-column tiles).
template <typename T>
struct EpiExpandRope {
  __device__ int b_row(int n) const { return n; }   // output column -> weight row
  static constexpr bool kWide = false;   // pair registers do not fit beside a 256x256 tile
  static constexpr bool kNarrow = false;
  T* kv; KvStrides ks; const float* bias; const float* sigma; int mode; const int* keep;
  T* kvo; KvStrides kso;   // destination when repairing out of place (kvo null: in place)
  const float2* rope;      // [M][head_dim/2] scaled (cos, sin)
  template <int COLS, int NT> struct Map {
    static constexpr int PAIRS = COLS / 16;        // 8-pair groups per tile row
    static constexpr int RSTEP = NT / PAIRS;
  };
  template <int ROWS, int COLS, int NT>
  struct Pre {
    static constexpr int P = ROWS / Map<COLS, NT>::RSTEP;
    float b1[8], b2[8], s1[8], s2[8];
    Vec8<T> x1[P], x2[P];
    int kp[P];
  };
  struct Cols { int c1, c2, i0; bool is_k, on; T* b1; T* o1; };
  template <int COLS, int NT>
  __device__ bool cols(int n0, int N, Cols& k) const {
    const int dh = ks.head_dim, half = dh / 2, sph = half / 8;
    const int p = threadIdx.x % Map<COLS, NT>::PAIRS;
    k.c1 = (p / sph) * dh + (p % sph) * 8;
    k.c2 = k.c1 + half;
    if (n0 + k.c2 >= N) return false;
    k.b1 = kv_coord(kv, ks, n0 + k.c1, &k.is_k);
    bool dummy;
    k.o1 = kvo ? kv_coord(kvo, kso, n0 + k.c1, &dummy) : k.b1;
    k.i0 = (n0 + k.c1) % dh;
    k.on = mode & (k.is_k ? EXPAND_K : EXPAND_V);
    return k.on || k.is_k || kvo;                  // stale V in place: nothing to write
  }
  template <int ROWS, int COLS, int NT>
  __device__ void prefetch(Pre<ROWS, COLS, NT>& p, int m0, int n0, int M, int N) const {
    Cols k;
    if (!cols<COLS, NT>(n0, N, k)) return;
    const int half = ks.head_dim / 2;
    load8f(bias + n0 + k.c1, p.b1); load8f(bias + n0 + k.c2, p.b2);
    load8f(sigma + n0 + k.c1, p.s1); load8f(sigma + n0 + k.c2, p.s2);
#pragma unroll
    for (int q = 0; q < Pre<ROWS, COLS, NT>::P; ++q) {
      const int gm = m0 + threadIdx.x / Map<COLS, NT>::PAIRS + q * Map<COLS, NT>::RSTEP;
      p.kp[q] = (gm < M && keep) ? keep[gm] : 0;
      if (gm < M) {
        const int64_t to = ks.tok(gm);
        p.x1[q].load(k.b1 + to);
        p.x2[q].load(k.b1 + half + to);
      }
    }
  }
  template <int ROWS, int COLS, int LDC, int NT>
  __device__ void run(const float* Cs, Pre<ROWS, COLS, NT>& p, int m0, int n0, int M, int N) const {
    Cols k;
    if (!cols<COLS, NT>(n0, N, k)) return;
    const int half = ks.head_dim / 2;
    constexpr int P = Pre<ROWS, COLS, NT>::P;
    const bool res = mode & EXPAND_RESIDUAL;
    constexpr int GRP = P >= 2 ? 2 : P;             // passes whose (cos, sin) load together
#pragma unroll
    for (int q0 = 0; q0 < P; q0 += GRP) {
    float4 cs[GRP][4];
    if (k.is_k) {
#pragma unroll
      for (int u = 0; u < GRP; ++u) {
        const int gm =
            min(m0 + (int)threadIdx.x / Map<COLS, NT>::PAIRS + (q0 + u) * Map<COLS, NT>::RSTEP, M - 1);
        const float4* t4 = reinterpret_cast<const float4*>(rope + (int64_t)gm * half + k.i0);
#pragma unroll
        for (int e = 0; e < 4; ++e) cs[u][e] = t4[e];
      }
    }
#pragma unroll
    for (int u = 0; u < GRP; ++u) {
      const int q = q0 + u;
      const int r = threadIdx.x / Map<COLS, NT>::PAIRS + q * Map<COLS, NT>::RSTEP, gm = m0 + r;
      if (gm >= M) continue;
      float y1[8], y2[8];
      p.x1[q].to_float(y1);
      p.x2[q].to_float(y2);
      if (k.on && !p.kp[q]) {
        float a1[8], a2[8];
        load8f(Cs + r * LDC + k.c1, a1);
        load8f(Cs + r * LDC + k.c2, a2);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          y1[e] = (res ? y1[e] : 0.f) + p.s1[e] * (a1[e] + p.b1[e]);
          y2[e] = (res ? y2[e] : 0.f) + p.s2[e] * (a2[e] + p.b2[e]);
        }
      } else if (!k.is_k && !kvo) {
        continue;
      }
      if (k.is_k) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float4 t = cs[u][e];   // (cos, sin) of pairs 2e and 2e+1
          const float u0 = y1[2 * e], v0 = y2[2 * e], u1 = y1[2 * e + 1], v1 = y2[2 * e + 1];
          y1[2 * e] = t.x * u0 - t.y * v0;
          y2[2 * e] = t.x * v0 + t.y * u0;
          y1[2 * e + 1] = t.z * u1 - t.w * v1;
          y2[2 * e + 1] = t.z * v1 + t.w * u1;
        }
      }
      p.x1[q].from_float(y1);
      p.x2[q].from_float(y2);
      const int64_t to = kvo ? kso.tok(gm) : ks.tok(gm);
      p.x1[q].store(k.o1 + to);
      p.x2[q].store(k.o1 + half + to);
    }
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

// Tile of this workgroup.  Workgroups are dealt to the 8 XCDs round-robin
// (linear id i runs on XCD i % 8), and each XCD has its own L2, so ids are
// first regrouped so that each XCD receives a contiguous run of tiles, and
// runs are walked in groups of TILE_GROUP tile rows, column by column: the
// workgroups resident on one XCD share a few A row panels and B column
// panels instead of each XCD fetching every panel.
constexpr int TILE_GROUP = 8;
template <typename G>
__device__ __forceinline__ void tile_of(int M, int N, int& tm, int& tn) {
  const int gm = (M + G::BM - 1) / G::BM, gn = (N + G::BN - 1) / G::BN;
  const int total = gm * gn;
  int id = blockIdx.x;
  if (total % 8 == 0) id = (id % 8) * (total / 8) + id / 8;
  const int per_group = TILE_GROUP * gn;
  const int first = (id / per_group) * TILE_GROUP;
  const int rows = min(gm - first, TILE_GROUP);
  const int k = id % per_group;
  tm = first + k % rows;
  tn = k / rows;
}

// A split along K into two row-major matrices: columns [0, k1) of the
// product's A come from A (lda), columns [k1, K) from a2 (lda2), so that
// C = [A | a2] B^T needs no concatenated copy.  k1 is a multiple of the slab.
template <typename T>
struct ASplit {
  const T* a2 = nullptr;
  int64_t lda2 = 0;
  int k1 = 0;
};

template <typename T, typename G, typename Epi, bool SPLIT = false>
__global__ __launch_bounds__(G::NT) void gemm_nt_kernel(const T* __restrict__ A, int64_t lda,
                                                      const T* __restrict__ B, int64_t ldb,
                                                      int M, int N, int K, Epi epi,
                                                      ASplit<T> sp) {
  using MM = Mma32<T>;
  using frag = typename MM::frag;
  __shared__ __align__(1024) char smem[G::LDS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int tm, tn;
  tile_of<G>(M, N, tm, tn);
  const int m0 = tm * G::BM, n0 = tn * G::BN;
  const int kg = wave / (G::WGM * G::WGN), wv = wave % (G::WGM * G::WGN);
  const int wm = (wv / G::WGN) * G::WM, wn = (wv % G::WGN) * G::WN;

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
  // the same rows of the second A matrix, read from slab k1 / BK on
  const char* asrc2[SPLIT ? G::A_ROUNDS : 1];
  const int kt1 = SPLIT ? sp.k1 / G::BK : 0;
  if constexpr (SPLIT) {
#pragma unroll
    for (int r = 0; r < G::A_ROUNDS; ++r) {
      const int row = (r * G::NW + wave) * 8 + (lane >> 3);
      const int chunk = (lane & 7) ^ swz128(row);
      asrc2[r] = reinterpret_cast<const char*>(sp.a2 + (int64_t)min(m0 + row, M - 1) * sp.lda2) +
                 chunk * 16;
    }
  }
#pragma unroll
  for (int r = 0; r < G::B_ROUNDS; ++r) {
    const int row = (r * G::NW + wave) * 8 + (lane >> 3);
    const int chunk = (lane & 7) ^ swz128(row);
    bsrc[r] = reinterpret_cast<const char*>(B + (int64_t)epi.b_row(min(n0 + row, N - 1)) * ldb) +
              chunk * 16;
  }
  // DMA operation o (A rounds first, then B rounds) of slab kt into a stage
  auto dma_op = [&](int o, int kt, int stage) {
    char* base = smem + stage * G::STAGE_BYTES;
    if (o < G::A_ROUNDS) {
      const char* a = asrc[o] + kt * 128;
      if constexpr (SPLIT) {
        if (kt >= kt1) a = asrc2[o] + (kt - kt1) * 128;
      }
      dma16(a, base + (o * G::NW + wave) * 1024);
    } else {
      const int r = o - G::A_ROUNDS;
      dma16(bsrc[r] + kt * 128, base + G::BM * 128 + (r * G::NW + wave) * 1024);
    }
  };
  auto issue = [&](int kt, int stage) {
#pragma unroll
    for (int o = 0; o < G::OPS; ++o) dma_op(o, kt, stage);
  };
  // Spread issue (the 8-wave 128-row tiles, whose 4-slab rings give a refill
  // three iterations to land): the refill goes out in equal shares over the
  // slab's k-steps, each share after that step's fragment reads for the next
  // step (a DMA writes LDS, so the compiler keeps it behind every earlier
  // read) and among its products, instead of as a burst after the barrier.
  // Every
  // slab is loaded, past the end as a copy of the last slab into a stage
  // nobody reads again, so each iteration issues the same OPS operations and
  // waits for the same count.  (2-slab rings keep the burst: their refill
  // must land within the iteration.)
  constexpr bool SPREAD = G::BM <= 128 && G::NW == 8;

  // the epilogue's global loads (bias, residuals, the stale cache) go out
  // before the main loop and land while it runs
  // (a single staging pass: before the main loop, where they land while it
  // runs; two passes: before each pass, so the loop keeps its registers)
  constexpr int ER = G::EPI_ROWS;
  typename Epi::template Pre<ER, G::BN, G::NT> pre;
  if constexpr (G::EARLY || G::EARLY2) epi.template prefetch<ER, G::BN, G::NT>(pre, m0, n0, M, N);

  f32x16 acc[G::TM][G::TN];
#pragma unroll
  for (int i = 0; i < G::TM; ++i)
#pragma unroll
    for (int j = 0; j < G::TN; ++j) acc[i][j] = f32x16{};

  const int KT = K / G::BK;
#pragma unroll
  for (int st = 0; st < G::STAGES - 1; ++st) {
    if constexpr (SPREAD) issue(min(st, KT - 1), st);
    else if (st < KT) issue(st, st);
  }

  // fragment rows: wm + i*32 + (lane & 31); all share swizzle ((lane & 15) >> 1)
  const int fr = lane & 31, fsw = (lane & 15) >> 1;
  for (int kt = 0; kt < KT; ++kt) {
    if constexpr (SPREAD) wait_vmcnt<G::OPS * (G::STAGES - 2)>();
    else wait_slab<G::OPS, G::STAGES - 2>(min(G::STAGES - 2, KT - 1 - kt));
    __builtin_amdgcn_s_barrier();
    const int nkt = min(kt + G::STAGES - 1, KT - 1), nst = (kt + G::STAGES - 1) % G::STAGES;
    if constexpr (!SPREAD) {
      if (kt + G::STAGES - 1 < KT) issue(nkt, nst);
    }

    const char* as = smem + (kt % G::STAGES) * G::STAGE_BYTES;
    const char* bs = as + G::BM * 128;
    // fragments double-buffered across the slab's k-steps: the reads of step
    // ks + 1 are issued between the products of step ks
    constexpr int NKS = G::BK / MM::KSTEP / G::KS;   // k-steps of this wave group
    const int ks0 = kg * NKS;
    frag af[2][G::TM], bfr[2][G::TN];
    auto ld = [&](int ks, int buf) {
      const int k = (ks0 + ks) * MM::KSTEP + (lane >> 5) * MM::KPL;
      const int cofs = (((k / G::VEC) ^ fsw) << 4) + (k % G::VEC) * (int)sizeof(T);
#pragma unroll
      for (int i = 0; i < G::TM; ++i)
        af[buf][i] = *reinterpret_cast<const frag*>(as + (wm + i * 32 + fr) * 128 + cofs);
#pragma unroll
      for (int j = 0; j < G::TN; ++j)
        bfr[buf][j] = *reinterpret_cast<const frag*>(bs + (wn + j * 32 + fr) * 128 + cofs);
    };
    ld(0, 0);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      if (ks + 1 < NKS) ld(ks + 1, (ks + 1) & 1);
#pragma unroll
      for (int i = 0; i < G::TM; ++i)
#pragma unroll
        for (int j = 0; j < G::TN; ++j)
          acc[i][j] = MM::mma(bfr[ks & 1][j], af[ks & 1][i], acc[i][j]);
      if constexpr (SPREAD) {
        // this k-step's share of the refill (after the next step's reads)
#pragma unroll
        for (int o = ks * G::OPS / NKS; o < (ks + 1) * G::OPS / NKS; ++o) dma_op(o, nkt, nst);
      }
    }
    // instruction order for the scheduler: the first step's LDS reads, then
    // every step's MFMAs alternating with the next step's reads (and, spread,
    // with its share of the next slab's DMA operations)
    constexpr int NR = G::TM + G::TN, NM = G::TM * G::TN;
    constexpr int NP = NR < NM ? NR : NM;
    __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);        // DS reads
#pragma unroll
    for (int ks = 0; ks + 1 < NKS; ++ks) {
#pragma unroll
      for (int r = 0; r < NP; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);       // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      if constexpr (NM > NP) __builtin_amdgcn_sched_group_barrier(0x008, NM - NP, 0);
      if constexpr (NR > NP) __builtin_amdgcn_sched_group_barrier(0x100, NR - NP, 0);
      // (spread: this step's share of the refill after its reads and products)
      if constexpr (SPREAD) {
        const int share = (ks + 1) * G::OPS / NKS - ks * G::OPS / NKS;
        for (int o = 0; o < share; ++o) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      }
    }
    if constexpr (SPREAD) {
      // the last step reads nothing; its products carry its share of the DMA
      constexpr int LAST = G::OPS - (NKS - 1) * G::OPS / NKS;
#pragma unroll
      for (int r = 0; r < NM; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        constexpr int DQ = LAST / NM, DR = LAST % NM;   // DMA ops per product
        if (r < DR) __builtin_amdgcn_sched_group_barrier(0x020, DQ + 1, 0);
        else if constexpr (DQ > 0) __builtin_amdgcn_sched_group_barrier(0x020, DQ, 0);
      }
    } else {
      __builtin_amdgcn_sched_group_barrier(0x008, NM, 0);
    }
  }
  // the copies past the last slab land in the ring, which the epilogue reuses
  if constexpr (SPREAD) wait_vmcnt<0>();

  // Epilogue.  With the weight tile as the MFMA's first operand, lane l of
  // atom (i, j) holds output row wm + i*32 + (l & 31) and, in registers
  // 4g .. 4g+3, the consecutive columns wn + j*32 + 8g + 4*(l >> 5) + [0, 4).
  // The tile is staged EPI_ROWS rows at a time with 16-byte LDS writes over
  // the ring, each pass after its epilogue loads have been issued.
  float* Cs = reinterpret_cast<float*>(smem);
  if constexpr (G::KS == 2) {
    // group 1 stages its partial tile; group 0 adds it to its own
    // accumulators (always group 0 + group 1) and stages the sum over it
    __syncthreads();  // ring no longer read
    auto stage = [&](bool add) {
#pragma unroll
      for (int i = 0; i < G::TM; ++i)
#pragma unroll
        for (int j = 0; j < G::TN; ++j)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            float4* c = reinterpret_cast<float4*>(Cs + (wm + i * 32 + fr) * G::LDC + wn + j * 32 +
                                                  g * 8 + (lane >> 5) * 4);
            float4 v = make_float4(acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                                   acc[i][j][4 * g + 3]);
            if (add) {
              const float4 o = *c;
              v = make_float4(v.x + o.x, v.y + o.y, v.z + o.z, v.w + o.w);
            }
            *c = v;
          }
    };
    if (kg == 1) stage(false);
    __syncthreads();
    if (kg == 0) stage(true);
    __syncthreads();
    epi.template run<ER, G::BN, G::LDC, G::NT>(Cs, pre, m0, n0, M, N);
    return;
  }
  // the accumulator rows of staging pass `part`, written over the ring (or
  // the previous pass's rows) once nobody reads it
  auto stage = [&](int part) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < G::TM; ++i) {
      const int r0 = wm + i * 32 - part * ER;   // first row of atom row i in this pass
      if (r0 < 0 || r0 >= ER) continue;
#pragma unroll
      for (int j = 0; j < G::TN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g)
          *reinterpret_cast<float4*>(Cs + (r0 + fr) * G::LDC + wn + j * 32 + g * 8 +
                                     (lane >> 5) * 4) =
              make_float4(acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                          acc[i][j][4 * g + 3]);
    }
    __syncthreads();
  };
#pragma unroll
  for (int part = 0; part < G::BM / ER; ++part) {
    if (part > 0 || !(G::EARLY || G::EARLY2))
      epi.template prefetch<ER, G::BN, G::NT>(pre, m0 + part * ER, n0, M, N);
    stage(part);
    epi.template run<ER, G::BN, G::LDC, G::NT>(Cs, pre, m0 + part * ER, n0, M, N);
  }
}

template <typename T, typename G, typename Epi, bool SPLIT = false>
static hipError_t launch_tiled(const T* A, int64_t lda, const T* B, int64_t ldb, int M, int N,
                               int K, const Epi& epi, hipStream_t s, ASplit<T> sp = {}) {
  if (M <= 0 || N <= 0) return hipSuccess;
  // the main loop streams whole 128-byte K slabs with 16-byte copies
  if (K <= 0 || K % G::BK != 0 || lda % G::VEC != 0 || ldb % G::VEC != 0 ||
      reinterpret_cast<uintptr_t>(A) % 16 != 0 || reinterpret_cast<uintptr_t>(B) % 16 != 0)
    return hipErrorInvalidValue;
  if (SPLIT && (!sp.a2 || sp.k1 <= 0 || sp.k1 >= K || sp.k1 % G::BK != 0 ||
                sp.lda2 % G::VEC != 0 || reinterpret_cast<uintptr_t>(sp.a2) % 16 != 0))
    return hipErrorInvalidValue;
  const int64_t tiles = (int64_t)((N + G::BN - 1) / G::BN) * ((M + G::BM - 1) / G::BM);
  if (tiles >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  dim3 grid((unsigned)tiles);
  CR_LAUNCH((gemm_nt_kernel<T, G, Epi, SPLIT>), grid, dim3(G::NT), 0, s, A, lda, B, ldb, M, N, K,
            epi, sp);
  return hipGetLastError();
}

// Tile choice.  bf16 products whose 256x256 tiling fills its rounds well
// enough (round_fill, kWideGain) take 256x256 tiles of eight waves
// (128x64 each, two per SIMD): half the operand bytes per FLOP of a 128x128
// tile, and one workgroup per CU with a two-slab ring of 64 KB slabs.
// Otherwise 128x128 tiles: grids of more than one workgroup per CU use four
// waves (64x64 each) and a two-slab ring (64 KB, two workgroups resident per
// CU hide each other's latency); grids that fit in one pass over the 256 CUs
// use eight waves (64x32 each, so two per SIMD) and a four-slab ring (three
// slabs in flight cover the fetch latency).  Epi::kWide is false for
// epilogues that need a 128-column tile or more registers than the 256x256
// tile leaves.
// Fraction of the workgroup slots busy over the rounds a grid of `tiles`
// takes on `slots` resident workgroups.
static inline double round_fill(int64_t tiles, int64_t slots) {
  const int64_t rounds = (tiles + slots - 1) / slots;
  return rounds > 0 ? (double)tiles / (double)(rounds * slots) : 0.0;
}
// A 256-row tile's main loop moves about 1.25x the FLOPs of a 128x128 tile
// per unit time (half the operand bytes per FLOP), so it is taken when that
// outweighs a worse fill of the last round.
constexpr double kWideGain = 1.25;

template <typename T, typename Epi, bool SPLIT = false>
static hipError_t launch(const T* A, int64_t lda, const T* B, int64_t ldb, int M, int N, int K,
                         const Epi& epi, hipStream_t s, ASplit<T> sp = {}) {
  if constexpr (sizeof(T) == 2 && Epi::kWide) {
    const int64_t wide_tiles = (int64_t)((M + 255) / 256) * ((N + 255) / 256);
    const int64_t tiles128 = (int64_t)((M + 127) / 128) * ((N + 127) / 128);
    const double fill128 = tiles128 <= 256 ? round_fill(tiles128, 256) : round_fill(tiles128, 512);
    if (kWideGain * round_fill(wide_tiles, 256) >= fill128)
      return launch_tiled<T, GemmTile<T, 4, 2, 2, 2, 4>, Epi, SPLIT>(A, lda, B, ldb, M, N, K, epi, s,
                                                                    sp);
  }
  const int64_t tiles = (int64_t)((M + 127) / 128) * ((N + 127) / 128);
  // Grids of at most half the CUs (short batches) take 64x64 tiles instead:
  // four times the workgroups (two resident per CU), each with a quarter of
  // the operand bytes per slab, on eight waves as two 4-wave K groups of
  // 32x32 waves.
  if constexpr (sizeof(T) == 2 && Epi::kNarrow) {
    if (tiles <= 128)
      return launch_tiled<T, GemmTile<T, 1, 1, 4, 2, 2, false, 2>, Epi, SPLIT>(A, lda, B, ldb, M, N,
                                                                              K, epi, s, sp);
  }
  if (tiles <= 256) {
    // long K: two 4-wave groups of 64x64 waves, each on half of every slab's
    // k-steps, read a third fewer fragment bytes from LDS per product than
    // eight waves of 64x32 (+3-4% at K = 2048-4096; at K = 1024 the extra
    // partial-tile sum costs more than it saves)
    if constexpr (sizeof(T) == 2) {
      if (K >= 2048)
        return launch_tiled<T, GemmTile<T, 2, 2, 4, 2, 2, false, 2>, Epi, SPLIT>(A, lda, B, ldb, M, N,
                                                                                K, epi, s, sp);
    }
    return launch_tiled<T, GemmTile<T, 2, 1, 4, 2, 4>, Epi, SPLIT>(A, lda, B, ldb, M, N, K, epi, s,
                                                                 sp);
  }
  return launch_tiled<T, GemmTile<T, 2, 2, 2>, Epi, SPLIT>(A, lda, B, ldb, M, N, K, epi, s, sp);
}

template <typename T>
hipError_t gemm_bias(const T* A, int64_t lda, const T* B, int64_t ldb, int M, int N, int K,
                     T* out, int64_t ldo, const float* bias, const T* resid, int64_t ldr,
                     bool gelu, hipStream_t s, const T* resid2, int64_t ldr2) {
  EpiBias<T> e{out, ldo, bias, resid, ldr, resid2, ldr2, gelu ? 1 : 0};
  return launch<T>(A, lda, B, ldb, M, N, K, e, s);
}

template <typename T>
hipError_t gemm_bias_split(const T* A, int64_t lda, int K1, const T* A2, int64_t lda2, const T* B,
                           int64_t ldb, int M, int N, int K, T* out, int64_t ldo,
                           const float* bias, const T* resid, int64_t ldr, hipStream_t s) {
  EpiBias<T> e{out, ldo, bias, resid, ldr, nullptr, 0, 0};
  return launch<T, EpiBias<T>, true>(A, lda, B, ldb, M, N, K, e, s, ASplit<T>{A2, lda2, K1});
}

template <typename T>
hipError_t gemm_qkv(const T* A, int64_t lda, const T* B, int M, int K, int d_b, int d_head,
                    T* q, T* k, T* vt, int64_t n_pad, const float* bias, const float2* rope,
                    hipStream_t s) {
  const int N = 3 * d_b;
  // 192-column tiles of whole heads on a 256x192 grid (eight waves of 64x96)
  // when it fills its rounds well enough; otherwise 128x128 tiles in the
  // weights' own column order.  Either grid covers rows up to roundup(M, 128)
  // >= n_pad, so the transposed V padding is written too (A rows >= M are
  // clamped copies: finite).
  if constexpr (sizeof(T) == 2) {
    const int64_t wide = (int64_t)((M + 255) / 256) * (N / 192);
    const int64_t tiles128 = (int64_t)((M + 127) / 128) * (N / 128);
    const double fill128 = tiles128 <= 256 ? round_fill(tiles128, 256) : round_fill(tiles128, 512);
    if (192 % (3 * d_head) == 0 && N % 192 == 0 && kWideGain * round_fill(wide, 256) >= fill128) {
      EpiQKVh<T> e{q, k, vt, n_pad, d_b, d_head, bias, rope};
      return launch_tiled<T, GemmTile<T, 2, 3, 2, 4, 2>>(A, lda, B, K, M, N, K, e, s);
    }
  }
  EpiQKV<T> e{q, k, vt, n_pad, d_b, d_head, bias, rope};
  return launch<T>(A, lda, B, K, M, N, K, e, s);
}

template <typename T>
hipError_t gemm_expand(const T* A, int64_t lda, const T* B, int M, int N, int K, T* kv,
                       KvStrides ks, const float* bias, const float* sigma, int mode,
                       const int* keep, const float2* key_rope, T* kv_out, KvStrides ks_out,
                       hipStream_t s) {
  if (key_rope) {
    if (ks.head_dim > 128) return hipErrorInvalidValue;
    if (128 % ks.head_dim == 0) {
      // a tile holds whole heads: the rotation is fused into the output add
      EpiExpandRope<T> e{kv, ks, bias, sigma, mode, keep, kv_out, ks_out, key_rope};
      return launch<T>(A, lda, B, K, M, N, K, e, s);
    }
    // heads straddle tile boundaries (head_dim 96): output add, then the
    // rotation of every key head of the written cache
    EpiExpand<T> e{kv, ks, bias, sigma, mode, keep, kv_out, ks_out};
    hipError_t err = launch<T>(A, lda, B, K, M, N, K, e, s);
    if (err != hipSuccess) return err;
    const KvStrides& kd = kv_out ? ks_out : ks;
    const int n_layers = N / (2 * ks.n_kv_heads * ks.head_dim);
    return rotate_keys<T>(kv_out ? kv_out : kv, kd, n_layers, M, key_rope, false, 1.0f, s);
  }
  EpiExpand<T> e{kv, ks, bias, sigma, mode, keep, kv_out, ks_out};
  if constexpr (sizeof(T) == 2) {
    const int64_t wide = (int64_t)((M + 255) / 256) * ((N + 255) / 256);
    const int64_t tiles128 = (int64_t)((M + 127) / 128) * ((N + 127) / 128);
    const double fill128 = tiles128 <= 256 ? round_fill(tiles128, 256) : round_fill(tiles128, 512);
    // the expansion's epilogue (the stale-cache read-modify-write) gains less
    // from the wide tile than the bias epilogues: about 5% at equal fill
    constexpr double kExpandWideGain = 1.05;
    if (kExpandWideGain * round_fill(wide, 256) >= fill128)
      return launch_tiled<T, GemmTile<T, 4, 2, 2, 2, 4, true>>(A, lda, B, K, M, N, K, e, s);
  }
  return launch<T>(A, lda, B, K, M, N, K, e, s);
}

#define CR_INST(T)                                                                              \
  template hipError_t gemm_bias<T>(const T*, int64_t, const T*, int64_t, int, int, int, T*,    \
                                   int64_t, const float*, const T*, int64_t, bool, hipStream_t, \
                                   const T*, int64_t);                                          \
  template hipError_t gemm_bias_split<T>(const T*, int64_t, int, const T*, int64_t, const T*,   \
                                         int64_t, int, int, int, T*, int64_t, const float*,      \
                                         const T*, int64_t, hipStream_t);                        \
  template hipError_t gemm_qkv<T>(const T*, int64_t, const T*, int, int, int, int, T*, T*, T*, \
                                  int64_t, const float*, const float2*, hipStream_t);            \
  template hipError_t gemm_expand<T>(const T*, int64_t, const T*, int, int, int, T*, KvStrides, \
                                     const float*, const float*, int, const int*,               \
                                     const float2*, T*, KvStrides, hipStream_t);
CR_INST(bf16)
CR_INST(float)
#undef CR_INST

}  // namespace cr
