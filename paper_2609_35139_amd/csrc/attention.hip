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
// A workgroup owns 128 queries of one head (32 per wave; 64 queries for
// grids too small to fill the chip, see below).  Scores are formed
// transposed, S^T = K Q^T, with 32x32 MFMA atoms, so that each lane holds the
// scores of one query: the online-softmax max and sum are register
// reductions plus one in-register exchange with lane ^ 32.  The K rows of
// each 32-key sub-tile are fed to the MFMA in an order (bits 2 and 3 of the
// row index swapped) that makes the score accumulator registers coincide
// with the B operand of the P V product, so probabilities never leave
// registers.
// V arrives transposed (vt[head][d][token]) from the QKV epilogue, so the
// A operand of O^T = V^T P^T is a contiguous 16-byte read.  K and V^T tiles
// stream through a four-stage LDS ring filled by global_load_lds.  The
// softmax keeps a per-row reference max that is not a running max: the
// score accumulators start at minus the reference, and the exact tile max is
// taken (with a rescale of the output accumulators) only for a row's first
// keys or when a tile's probability sum exceeds 2^24, a choice made row by
// row.  Softmax is invariant to the reference, so this changes rounding
// only, and per score the VALU does an exp2, half a pack and half a dot2
// instead of also a max and a subtraction.
#include <climits>
#include <type_traits>

#include "launch.h"

namespace cr {

// largest tile row sum accepted without re-deriving the reference max
constexpr float kMaxTileSum = 16777216.0f;   // 2^24

// Eight waves per workgroup in GROUPS = 8 / WPG groups of WPG waves: a
// workgroup owns BQ = 32 * WPG queries, and the groups split its key tiles.
template <typename T, int D, int STAGES_ = 4, int WPG_ = 4>
struct AttnCfg {
  static constexpr int WPG = WPG_, BQ = 32 * WPG, BKV = 64, STAGES = STAGES_;
  static constexpr int GROUPS = 8 / WPG, NT = 512;
  static constexpr int VEC = 16 / (int)sizeof(T);
  static constexpr int RBK = D * (int)sizeof(T);      // K tile row bytes
  static constexpr int RBV = BKV * (int)sizeof(T);    // V^T tile row bytes
  static constexpr int K_BYTES = BKV * RBK, V_BYTES = D * RBV;
  // a group's waves fill 1 KB each per DMA round
  static constexpr int K_ROUNDS = K_BYTES / (WPG * 1024), V_ROUNDS = V_BYTES / (WPG * 1024);
  static constexpr int OPS = K_ROUNDS + V_ROUNDS;     // DMA ops per thread per tile
  static constexpr int STAGE_BYTES = K_BYTES + V_BYTES;
  static constexpr int RING_BYTES = STAGES * STAGE_BYTES;
  // merge area: each group but the first hands (m, l, O^T) of its BQ
  // queries to group 0; rows of D + 1 floats, so the 32 queries of a wave
  // fall in distinct banks
  static constexpr int MLD = D + 1;
  static constexpr int MERGE_ONE = BQ * MLD * 4 + 2 * BQ * 2 * 4;
  static constexpr int MERGE_BYTES = (GROUPS - 1) * MERGE_ONE;
  static_assert(GROUPS * WPG == 8 && K_ROUNDS * WPG * 1024 == K_BYTES &&
                V_ROUNDS * WPG * 1024 == V_BYTES, "wave groups");
  static constexpr int LDS = GROUPS * RING_BYTES > MERGE_BYTES ? GROUPS * RING_BYTES : MERGE_BYTES;
};

// A-operand row r of a 32-key sub-tile reads key swap_bits23(r).
__device__ __forceinline__ int swap_bits23(int r) {
  return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1);
}
// Key (within a 32-key sub-tile) held by score register i of lane half g.
__device__ __forceinline__ int score_key(int g, int i) { return (i >> 3) * 16 + g * 8 + (i & 7); }

// Two groups of four waves share the 128 queries of a workgroup and split
// its key tiles (group g takes tiles g, g + 2, ...), each with its own online
// softmax state and LDS ring; group 1's partial result is merged into group
// 0's at the end.  This halves the critical path of the long query tiles of
// late chunks and keeps two waves per SIMD so that one wave's softmax
// overlaps the other's MFMAs.  A grid of fewer workgroups than half the CUs
// (a short batch) instead takes 64-query tiles with four groups of two
// waves (tiles g, g + 4, ...; two-slot rings, merged in group order): twice
// the workgroups, each group walking a quarter of the key tiles.
//
// Q arrives pre-scaled by log2(e)/sqrt(d_head) (QKV epilogue), so scores are
// in exp2 units.  K and V^T are padded with finite rows up to n_pad, so tile
// loads need no clamping.  The tile loop is unrolled over the STAGES ring
// slots: every LDS address is a per-lane base plus a compile-time offset.
template <typename T, int D, int STAGES = 4, int WPG = 4>
__global__ __launch_bounds__(512) void attention_kernel(const T* __restrict__ Q,
                                                        const T* __restrict__ Kg,
                                                        const T* __restrict__ Vt,
                                                        T* __restrict__ O, int N, int d_b,
                                                        int n_heads, int64_t n_pad,
                                                        const int* __restrict__ lo_arr,
                                                        const int* __restrict__ hi_arr,
                                                        int n_qtiles) {
  using C = AttnCfg<T, D, STAGES, WPG>;
  using MM = Mma32<T>;
  using frag = typename MM::frag;
  using SK = Swz<C::RBK>;
  using SV = Swz<C::RBV>;
  constexpr int KPL = MM::KPL, KSTEP = MM::KSTEP;
  constexpr int QF = D / KSTEP;          // Q fragments per lane
  constexpr int DT = D / 32;             // 32-row tiles of O^T
  constexpr int PS = 32 / KSTEP;         // P fragments per 32-key sub-tile
  __shared__ __align__(1024) char lds[C::LDS];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave / WPG, gw = wave % WPG;
  const int g = lane >> 5, ql = lane & 31;
  const int head = blockIdx.x % n_heads;
  const int qt = n_qtiles - 1 - blockIdx.x / n_heads;   // latest (longest) tiles first
  const int q = qt * C::BQ + gw * 32 + ql;
  const bool qvalid = q < N;
  char* ring = lds + grp * C::RING_BYTES;

  // Rows are tokens in order and lo, hi never decrease with the row (each is
  // the start or end of the row's request or chunk, or the row + 1), so the
  // workgroup's key range [lo(first row), hi(last row)) and the window that
  // every row of a wave admits, [lo(its last row), hi(its first row)), are
  // read from the end rows: uniform loads, no reductions, no barrier.
  const int q0 = qt * C::BQ, q1 = min(q0 + C::BQ, N) - 1;
  const int w0 = q0 + gw * 32, w1 = min(w0 + 32, N) - 1;
  const int kv_begin = lo_arr[q0], kv_end = hi_arr[q1];
  const int wmax_lo = w0 < N ? lo_arr[w1] : INT_MIN;
  const int wmin_hi = w0 < N ? hi_arr[w0] : INT_MAX;
  const int mlo = qvalid ? lo_arr[q] : INT_MIN, mhi = qvalid ? hi_arr[q] : INT_MAX;
  const int kb = (kv_begin / C::BKV) * C::BKV;
  const int ntiles = (kv_end - kb + C::BKV - 1) / C::BKV;
  const int iters = (ntiles + C::GROUPS - 1) / C::GROUPS;          // tiles per group
  const int mine = (ntiles - grp + C::GROUPS - 1) / C::GROUPS;     // tiles this group owns

  // Q^T fragments stay in registers: col = query, k = d
  frag qf[QF];
#pragma unroll
  for (int s = 0; s < QF; ++s) {
    if (qvalid) qf[s] = load_frag<T, frag>(Q + (int64_t)q * d_b + head * D + s * KSTEP + g * KPL);
    else qf[s] = frag{};
  }

  // DMA sources (per lane) of the workgroup's first key tile: K rows are
  // keys, V^T rows are d.  Both are padded to n_pad >= roundup(N, 64) keys.
  const char* ksrc[C::K_ROUNDS];
  const char* vsrc[C::V_ROUNDS];
#pragma unroll
  for (int r = 0; r < C::K_ROUNDS; ++r) {
    const int row = (r * WPG + gw) * SK::RPW + lane / SK::CPR;
    const int chunk = SK::slot(row, lane % SK::CPR);
    ksrc[r] = reinterpret_cast<const char*>(Kg + (int64_t)(kb + row) * d_b + head * D) + chunk * 16;
  }
#pragma unroll
  for (int r = 0; r < C::V_ROUNDS; ++r) {
    const int row = (r * WPG + gw) * SV::RPW + lane / SV::CPR;
    const int chunk = SV::slot(row, lane % SV::CPR);
    vsrc[r] = reinterpret_cast<const char*>(Vt + ((int64_t)head * D + row) * n_pad + kb) + chunk * 16;
  }
  const int64_t ktile_bytes = (int64_t)C::BKV * d_b * sizeof(T);

  // per-lane LDS read addresses inside slot 0 of the ring: K fragment kk of
  // sub-tile 0 (sub-tile 1 is 32 rows further; the swizzle is periodic in 32
  // rows), and the V^T fragment of sub-tile rt, P fragment s2 (dt adds 32 rows)
  const int krow = swap_bits23(ql);
  const char* kp[QF];
#pragma unroll
  for (int kk = 0; kk < QF; ++kk) {
    const int k = kk * KSTEP + g * KPL;
    kp[kk] = ring + SK::offset(krow, k / C::VEC) + (k % C::VEC) * (int)sizeof(T);
  }
  const char* vp[2][PS];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int s2 = 0; s2 < PS; ++s2) {
      const int kofs = rt * 32 + score_key(g, s2 * KPL);
      vp[rt][s2] = ring + C::K_BYTES + SV::offset(ql, kofs / C::VEC) + (kofs % C::VEC) * (int)sizeof(T);
    }

  f32x16 oacc[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d) oacc[d] = f32x16{};
  // m_ref: the row's reference max (exp2 units), shared by both lane halves
  // of a query; negm holds -m_ref (0 while there is none) as the score
  // accumulators' initial value
  float m_ref = -INFINITY, lsum = 0.f;
  f32x16 negm;
#pragma unroll
  for (int i = 0; i < 16; ++i) negm[i] = 0.f;

  // group-local tile i (workgroup tile 2i + grp) into ring slot SLOT
  auto issue = [&](int i, int slot_bytes) {
    char* base = ring + slot_bytes;
    const int64_t tile = (int64_t)C::GROUPS * i + grp;
#pragma unroll
    for (int r = 0; r < C::K_ROUNDS; ++r)
      dma16(ksrc[r] + tile * ktile_bytes, base + (r * WPG + gw) * 1024);
#pragma unroll
    for (int r = 0; r < C::V_ROUNDS; ++r)
      dma16(vsrc[r] + tile * C::BKV * (int64_t)sizeof(T), base + C::K_BYTES + (r * WPG + gw) * 1024);
  };

  // one key tile held in ring slot J (compile time)
  auto step = [&](auto slot, int it) {
    constexpr int J = decltype(slot)::value;
    if (it >= iters) return;
    // every iteration issues one tile (past the group's last tile, a copy of
    // it into a slot nobody reads again), so tile `it` has landed once
    // STAGES-2 later ones remain in flight
    wait_vmcnt<(C::STAGES - 2) * C::OPS>();
    __builtin_amdgcn_s_barrier();   // the slot refilled below is no longer read by anyone
    if (it >= mine) return;         // a group without a tile this round: only keeps the barrier count
    constexpr int SO = J * C::STAGE_BYTES;
    // the compiler's interleaving of LDS reads with MFMAs for this tile's
    // fragment reads and score products (-2% per launch, same results)
    __builtin_amdgcn_iglp_opt(0);

    // S^T = K Q^T for two 32-key sub-tiles; all fragment reads first
    frag kf[2][QF];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int kk = 0; kk < QF; ++kk)
        kf[rt][kk] = *reinterpret_cast<const frag*>(kp[kk] + (SO + rt * 32 * C::RBK));
    // V^T fragments of this tile for O^T += V^T P^T, read before the score
    // products so that their LDS latency hides behind the MFMAs and softmax
    // (bf16; the fp32 fragments are too many registers to hold that long)
    constexpr bool kEarlyV = sizeof(T) == 2;
    frag vf[2][PS][DT];
    auto read_v = [&] {
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int s2 = 0; s2 < PS; ++s2)
#pragma unroll
          for (int d = 0; d < DT; ++d)
            vf[rt][s2][d] = *reinterpret_cast<const frag*>(vp[rt][s2] + (SO + d * 32 * C::RBV));
    };
    if constexpr (kEarlyV) read_v();
    // the refill of the slot freed by the barrier goes out after this tile's
    // fragment reads (a DMA writes LDS, so the compiler keeps it behind every
    // earlier read), among the score products instead of ahead of them
    issue(min(it + C::STAGES - 1, mine - 1), ((J + C::STAGES - 1) % C::STAGES) * C::STAGE_BYTES);
    // the accumulators start at -m_use, so the scores arrive already shifted
    // by the row's reference max (no per-score subtraction)
    f32x16 s[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      s[rt] = MM::mma(kf[rt][0], qf[0], negm);
#pragma unroll
      for (int kk = 1; kk < QF; ++kk) s[rt] = MM::mma(kf[rt][kk], qf[kk], s[rt]);
    }
    const int k0 = kb + (C::GROUPS * it + grp) * C::BKV;
    if (!(k0 >= wmax_lo && k0 + C::BKV <= wmin_hi)) {
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = k0 + rt * 32 + score_key(g, i);
          if (key < mlo || key >= mhi) s[rt][i] = -INFINITY;
        }
    }
    // probabilities packed straight into the B operand of P V; the tile's
    // row sum is taken over the packed values the product uses
    frag pb[2][PS];
    auto probs = [&](auto shifted, float shift) {
      // one partial sum per fragment, so the dot2 chains are independent
      float tp[2][PS];
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int s2 = 0; s2 < PS; ++s2) {
          float pv[KPL];
#pragma unroll
          for (int e = 0; e < KPL; ++e)
            pv[e] = __builtin_amdgcn_exp2f(decltype(shifted)::value ? s[rt][s2 * KPL + e] - shift
                                                                    : s[rt][s2 * KPL + e]);
          pb[rt][s2] = pack_frag(pv, (frag*)nullptr);
          tp[rt][s2] = frag_sum(pb[rt][s2], 0.f);
        }
      float ts = 0.f;
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int s2 = 0; s2 < PS; ++s2) ts += tp[rt][s2];
      return ts;
    };
    // Fast path: the reference max stays where it is.  A probability is at
    // most its lane's tile sum, so a sum <= kMaxTileSum rules out overflow
    // (O and l accumulate in fp32 with ample range).  Otherwise, and for a
    // row without a reference yet, the row takes the exact row max, rescales
    // its accumulators and recomputes the tile's probabilities.  The choice
    // is made per query row (its two lanes agree through one exchange), so
    // no row's rounding depends on the scores of another row.  The fast
    // probabilities are skipped only when every row of the wave takes the
    // exact path anyway.
    float ts = 0.f;
    if (!__all(m_ref == -INFINITY)) ts = probs(std::false_type{}, 0.f);
    int exact = m_ref == -INFINITY || !(ts <= kMaxTileSum);
    exact = halves_or(exact);
    if (exact) {
      float mx = -INFINITY;
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[rt][i]);
      mx = halves_max(mx);
      const float m_use = m_ref == -INFINITY ? 0.f : m_ref;
      const float m_new = fmaxf(m_ref, mx + m_use);
      const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_ref - m_new);
      lsum *= alpha;
#pragma unroll
      for (int d = 0; d < DT; ++d)
#pragma unroll
        for (int i = 0; i < 16; ++i) oacc[d][i] *= alpha;
      m_ref = m_new;
      ts = probs(std::true_type{}, m_new == -INFINITY ? 0.f : m_new - m_use);
      const float nm = m_new == -INFINITY ? 0.f : -m_new;
#pragma unroll
      for (int i = 0; i < 16; ++i) negm[i] = nm;
    }
    lsum += ts;
    if constexpr (!kEarlyV) read_v();
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int s2 = 0; s2 < PS; ++s2)
#pragma unroll
        for (int d = 0; d < DT; ++d) oacc[d] = MM::mma(vf[rt][s2][d], pb[rt][s2], oacc[d]);
  };

#pragma unroll
  for (int st = 0; st < C::STAGES - 1; ++st)
    if (mine > 0) issue(min(st, mine - 1), st * C::STAGE_BYTES);
  for (int it0 = 0; it0 < iters; it0 += C::STAGES) {
    step(std::integral_constant<int, 0>{}, it0);
    step(std::integral_constant<int, 1>{}, it0 + 1);
    if constexpr (C::STAGES > 2) step(std::integral_constant<int, 2 % C::STAGES>{}, it0 + 2);
    if constexpr (C::STAGES > 3) step(std::integral_constant<int, 3 % C::STAGES>{}, it0 + 3);
  }

  // merge the other groups into group 0: per query q' = gw*32 + ql, lane half
  // g holds l (partial over its keys) and rows d = dt*32 + (v/4)*8 + g*4 + v%4
  // of O^T; group gi > 0 hands them over in merge region gi - 1
  wait_vmcnt<0>();   // the copies past the last tile land in the rings
  __syncthreads();   // every ring idle
  auto mo_of = [&](int gi) { return reinterpret_cast<float*>(lds + (gi - 1) * C::MERGE_ONE); };
  auto ml_of = [&](int gi) { return mo_of(gi) + C::BQ * C::MLD; };   // [BQ][2] (m, l) per half
  const int qrow = gw * 32 + ql;
  if (grp >= 1) {
    float* mo = mo_of(grp);
    float* ml = ml_of(grp);
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        mo[qrow * C::MLD + d * 32 + (v >> 2) * 8 + g * 4 + (v & 3)] = oacc[d][v];
    ml[(qrow * 2 + g) * 2 + 0] = m_ref;
    ml[(qrow * 2 + g) * 2 + 1] = lsum;
  }
  __syncthreads();
  if (grp >= 1 || !qvalid) return;
  T* orow = O + (int64_t)q * d_b + head * D;
  auto store4 = [&](int dd, const float* vals) {
    T outv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) outv[e] = from_f32<T>(vals[e]);
    if constexpr (sizeof(T) == 2) {
      *reinterpret_cast<uint2*>(orow + dd) = *reinterpret_cast<const uint2*>(outv);
    } else {
      *reinterpret_cast<uint4*>(orow + dd) = *reinterpret_cast<const uint4*>(outv);
    }
  };
  if constexpr (C::GROUPS == 2) {
    const float* mo = mo_of(1);
    const float* ml = ml_of(1);
    const float m1 = ml[(qrow * 2 + g) * 2 + 0], l1 = ml[(qrow * 2 + g) * 2 + 1];
    const float mt = fmaxf(m_ref, m1);
    const float a0 = m_ref == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_ref - mt);
    const float a1 = m1 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m1 - mt);
    const float lpart = lsum * a0 + l1 * a1;
    const float total = halves_sum(lpart);
    const float inv = 1.0f / total;
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int dd = d * 32 + i4 * 8 + g * 4;
        float vals[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          vals[e] = (oacc[d][i4 * 4 + e] * a0 + mo[qrow * C::MLD + dd + e] * a1) * inv;
        store4(dd, vals);
      }
  } else {
    // groups combined in index order with one common max
    float mg[C::GROUPS], lg[C::GROUPS], ag[C::GROUPS];
    mg[0] = m_ref;
    lg[0] = lsum;
#pragma unroll
    for (int gi = 1; gi < C::GROUPS; ++gi) {
      mg[gi] = ml_of(gi)[(qrow * 2 + g) * 2 + 0];
      lg[gi] = ml_of(gi)[(qrow * 2 + g) * 2 + 1];
    }
    float mt = mg[0];
#pragma unroll
    for (int gi = 1; gi < C::GROUPS; ++gi) mt = fmaxf(mt, mg[gi]);
    float lpart = 0.f;
#pragma unroll
    for (int gi = 0; gi < C::GROUPS; ++gi) {
      ag[gi] = mg[gi] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mg[gi] - mt);
      lpart += lg[gi] * ag[gi];
    }
    const float inv = 1.0f / halves_sum(lpart);
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int i4 = 0; i4 < 4; ++i4) {
        const int dd = d * 32 + i4 * 8 + g * 4;
        float vals[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float o = oacc[d][i4 * 4 + e] * ag[0];
#pragma unroll
          for (int gi = 1; gi < C::GROUPS; ++gi) o += mo_of(gi)[qrow * C::MLD + dd + e] * ag[gi];
          vals[e] = o * inv;
        }
        store4(dd, vals);
      }
  }
}

template <typename T>
hipError_t attention(const T* q, const T* k, const T* vt, T* o, int N, int d_b, int n_heads,
                     int d_head, int64_t n_pad, const int* lo, const int* hi, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  if (n_pad < ((N + 63) / 64) * 64) return hipErrorInvalidValue;
  const int n_qtiles = (N + 127) / 128;
  dim3 grid(n_qtiles * n_heads);
  // two rings (one per wave group) must fit in 160 KB of LDS
  constexpr int kStages = sizeof(T) == 2 ? 4 : 2;
  // A grid of fewer workgroups than half the CUs (short batches) takes
  // 64-query tiles whose four 2-wave groups split the key tiles (two-slot
  // rings): twice the workgroups, each with half the key tiles per group.
  if constexpr (sizeof(T) == 2) {
    if ((int64_t)n_qtiles * n_heads < 128) {
      const int n_q64 = (N + 63) / 64;
      dim3 g64(n_q64 * n_heads);
      if (d_head == 64) {
        CR_LAUNCH((attention_kernel<T, 64, 2, 2>), g64, dim3(512), 0, s, q, k, vt, o, N, d_b,
                  n_heads, n_pad, lo, hi, n_q64);
        return hipGetLastError();
      }
      if (d_head == 32) {
        CR_LAUNCH((attention_kernel<T, 32, 2, 2>), g64, dim3(512), 0, s, q, k, vt, o, N, d_b,
                  n_heads, n_pad, lo, hi, n_q64);
        return hipGetLastError();
      }
    }
  }
  if (d_head == 64) {
    CR_LAUNCH((attention_kernel<T, 64, kStages>), grid, dim3(512), 0, s, q, k, vt, o, N, d_b,
              n_heads, n_pad, lo, hi, n_qtiles);
  } else if (d_head == 32) {
    CR_LAUNCH((attention_kernel<T, 32, kStages>), grid, dim3(512), 0, s, q, k, vt, o, N, d_b,
              n_heads, n_pad, lo, hi, n_qtiles);
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
