// Row-wise and setup kernels of the repair forward pass (gfx950):
//  - LayerNorm with wavefront reductions (one wave per row),
//  - StaleEncoder stage 1 (per-segment projections streaming the cache),
//  - the chunk schedule of the block-causal mask,
//  - the RoPE (cos, sin) table,
//  - one-time weight preparation (transpose / widen).
#include <algorithm>
#include <cmath>
#include <vector>

#include "launch.h"

namespace cr {

__device__ __forceinline__ void load8(const float* p, float* v) {
  const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

// ------------------------------------------------------------- LayerNorm
// y = (x - mean) / sqrt(var + eps) * g + b over rows of C elements, biased
// variance, statistics in fp32 from values held in registers (two passes).
// A wave normalises R rows with one copy of gamma and beta in registers;
// every load (R rows, gamma, beta) is issued before the first reduction.
template <typename T, int MAXV, int R>
__global__ __launch_bounds__(256) void layernorm_kernel(const T* __restrict__ x, int64_t ldx,
                                                        T* __restrict__ y, int64_t ldy,
                                                        const float* __restrict__ g,
                                                        const float* __restrict__ b, int M,
                                                        int C, float eps) {
  const int lane = threadIdx.x & 63;
  const int row0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * R;
  if (row0 >= M) return;
  float v[R][MAXV][8], gv[MAXV][8], bv[MAXV][8];
#pragma unroll
  for (int k = 0; k < MAXV; ++k) {
    const int c = (k * 64 + lane) * 8;
    if (c < C) {
#pragma unroll
      for (int r = 0; r < R; ++r)
        if (row0 + r < M) { Vec8<T> t; t.load(x + (int64_t)(row0 + r) * ldx + c); t.to_float(v[r][k]); }
      load8(g + c, gv[k]);
      load8(b + c, bv[k]);
    }
  }
  float mean[R], rstd[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < MAXV; ++k)
      if ((k * 64 + lane) * 8 < C) {
#pragma unroll
        for (int e = 0; e < 8; ++e) sum += v[r][k][e];
      }
    mean[r] = wave_sum(sum) / (float)C;
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    float sq = 0.f;
#pragma unroll
    for (int k = 0; k < MAXV; ++k)
      if ((k * 64 + lane) * 8 < C) {
#pragma unroll
        for (int e = 0; e < 8; ++e) { const float d = v[r][k][e] - mean[r]; sq += d * d; }
      }
    rstd[r] = 1.0f / sqrtf(wave_sum(sq) / (float)C + eps);
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (row0 + r >= M) break;
    T* yr = y + (int64_t)(row0 + r) * ldy;
#pragma unroll
    for (int k = 0; k < MAXV; ++k) {
      const int c = (k * 64 + lane) * 8;
      if (c < C) {
        float o[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = (v[r][k][e] - mean[r]) * rstd[r] * gv[k][e] + bv[k][e];
        Vec8<T> t; t.from_float(o); t.store(yr + c);
      }
    }
  }
}

template <typename T>
hipError_t layernorm(const T* x, int64_t ldx, T* y, int64_t ldy, const float* g, const float* b,
                     int M, int C, float eps, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  // one row per wave: four resident workgroups per SIMD hide the reductions'
  // latency (several rows per wave with fewer waves measured slower)
  if (C <= 1024) {
    CR_LAUNCH((layernorm_kernel<T, 2, 1>), dim3((M + 3) / 4), dim3(256), 0, s, x, ldx, y, ldy,
              g, b, M, C, eps);
  } else {
    CR_LAUNCH((layernorm_kernel<T, 4, 1>), dim3((M + 3) / 4), dim3(256), 0, s, x, ldx, y, ldy,
              g, b, M, C, eps);
  }
  return hipGetLastError();
}

// ------------------------------------------------- StaleEncoder stage 1
// u_g = (x_g / sigma_g) W1_g + b1_g for every segment g = (l, kv, h), with
// 1/sigma folded into the prepared weights wseg[g][32][d_h] (rows >= d_seg
// are zero) and bseg[g][32].  One workgroup = TOK = 16*TB tokens x four
// consecutive segments (one per wave), so a workgroup streams whole runs of
// the cache rows and a wave's weight fragments serve TB token blocks.  The
// product is formed transposed, U^T = W X^T, on 16x16 MFMA atoms fed
// straight from the cache rows (every load is issued before the first
// product): a lane ends with four consecutive output columns of one token.
// The workgroup's outputs (4*d_seg contiguous columns per token) are staged
// in LDS and written as 16-byte row runs.
template <typename T, int DH, int TB>
__global__ __launch_bounds__(256) void compress_segments_kernel(
    const T* __restrict__ kv, KvStrides ks, const T* __restrict__ wseg,
    const float* __restrict__ bseg, T* __restrict__ U, int64_t ldu, int d_seg, int N, int S,
    int Kc) {
  using MM = Mma16<T>;
  using frag = typename MM::frag;
  constexpr int NK = DH / MM::KSTEP;
  constexpr int TOK = 16 * TB;
  constexpr int VE = 16 / (int)sizeof(T);
  // [token][4 segments x <= 32 columns]; rows padded by 16 bytes so that the
  // 16 tokens written together fall in distinct LDS banks
  constexpr int LDST = 128 + 16 / (int)sizeof(T);
  __shared__ __align__(16) T stage[TOK * LDST];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g0 = blockIdx.y * 4, g = g0 + wave;
  const int span = min(4, S - g0) * d_seg;
  const int t0 = blockIdx.x * TOK;
  const int fk = (lane >> 4) * MM::KPL;
  if (g < S) {
    const int h = g % ks.n_kv_heads, lk = g / ks.n_kv_heads;
    const T* base = kv + (int64_t)(lk >> 1) * ks.layer + (int64_t)(lk & 1) * ks.kv +
                    (int64_t)h * ks.head;
    const T* wg = wseg + (int64_t)g * 32 * DH;
    frag x[TB][NK], w[2][NK];
#pragma unroll
    for (int b = 0; b < TB; ++b) {
      const int t = t0 + b * 16 + (lane & 15);
#pragma unroll
      for (int k = 0; k < NK; ++k)
        x[b][k] = t < N ? load_frag<T, frag>(base + ks.tok(t) + k * MM::KSTEP + fk) : frag{};
    }
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int k = 0; k < NK; ++k)
        w[j][k] = load_frag<T, frag>(wg + (j * 16 + (lane & 15)) * DH + k * MM::KSTEP + fk);
    // output columns j*16 + (lane >> 4)*4 + e of token b*16 + (lane & 15)
    float bb[2][4];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = j * 16 + (lane >> 4) * 4 + e;
        bb[j][e] = c < d_seg ? bseg[g * 32 + c] : 0.f;
      }
#pragma unroll
    for (int b = 0; b < TB; ++b) {
      f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
      for (int k = 0; k < NK; ++k)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[j] = MM::mma(w[j][k], x[b][k], acc[j]);
      const int r = b * 16 + (lane & 15);
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int c = j * 16 + (lane >> 4) * 4 + e;
          if (c < d_seg) stage[r * LDST + wave * d_seg + c] = from_f32<T>(acc[j][e] + bb[j][e]);
        }
    }
  }
  __syncthreads();
  // token rows of `span` contiguous columns from column g0*d_seg
  const int64_t col0 = (int64_t)g0 * d_seg;
  if (span % VE == 0 && col0 % VE == 0) {
    const int cpr = span / VE;
    for (int i = threadIdx.x; i < TOK * cpr; i += 256) {
      const int r = i / cpr, c = (i % cpr) * VE, t = t0 + r;
      if (t < N)
        *reinterpret_cast<uint4*>(U + (int64_t)t * ldu + col0 + c) =
            *reinterpret_cast<const uint4*>(stage + r * LDST + c);
    }
  } else {
    for (int i = threadIdx.x; i < TOK * span; i += 256) {
      const int r = i / span, c = i % span, t = t0 + r;
      if (t < N) U[(int64_t)t * ldu + col0 + c] = stage[r * LDST + c];
    }
  }
  if (blockIdx.y == 0) {  // zero the K padding of U for these tokens
    const int pad = (int)(ldu - Kc);
    for (int idx = threadIdx.x; idx < TOK * pad; idx += 256) {
      const int t = t0 + idx / pad;
      if (t < N) U[(int64_t)t * ldu + Kc + idx % pad] = from_f32<T>(0.f);
    }
  }
}

template <typename T>
hipError_t compress_segments(const T* kv, KvStrides ks, int n_layers, const T* wseg,
                             const float* bseg, T* U, int64_t ldu, int d_seg, int N,
                             hipStream_t s) {
  if (N <= 0) return hipSuccess;
  const int S = 2 * n_layers * ks.n_kv_heads;
  // four 16-token blocks per wave (bf16) once the grid still fills the chip
  // several times over; one block otherwise and for fp32 (register budget)
  const bool wide = sizeof(T) == 2 && (int64_t)((N + 63) / 64) * ((S + 3) / 4) >= 1024;
#define CR_COMPRESS_TB(DH, TB)                                                                 \
  CR_LAUNCH((compress_segments_kernel<T, DH, TB>), dim3((N + 16 * TB - 1) / (16 * TB), (S + 3) / 4), \
            dim3(256), 0, s, kv, ks, wseg, bseg, U, ldu, d_seg, N, S, S * d_seg)
#define CR_COMPRESS(DH)                                                                        \
  case DH:                                                                                     \
    if (wide) CR_COMPRESS_TB(DH, (sizeof(T) == 2 ? 4 : 1));                                    \
    else CR_COMPRESS_TB(DH, 1);                                                                \
    break;
  switch (ks.head_dim) {
    CR_COMPRESS(32) CR_COMPRESS(64) CR_COMPRESS(96) CR_COMPRESS(128)
    CR_COMPRESS(160) CR_COMPRESS(192) CR_COMPRESS(224) CR_COMPRESS(256)
    default: return hipErrorInvalidValue;
  }
#undef CR_COMPRESS
#undef CR_COMPRESS_TB
  return hipGetLastError();
}

// ---------------------------------------------------------- chunk schedule
// Per token t: the key interval [lo, hi) of its attention row under the
// chosen topology (all of them allow only t's request), its 0-based position
// within the request, optionally its global position and a flag for the
// first chunk of its request, and optionally the repair network's RoPE row
// of that position (one row per token, so that the QKV epilogue's table
// reads do not wait for a position load first).  Chunks are passed by value
// in batches.  With the table, thread (t, i) handles pair i of token t and
// the threads with i = 0 write the schedule.
constexpr int SCHED_CHUNKS = 128;
struct SchedBatch {
  int count;                          // chunks in this batch
  int mask;                           // topology, values of CR_MASK_*
  int offs[SCHED_CHUNKS + 1];         // token offsets of the batch's chunks
  int req_start[SCHED_CHUNKS];        // first token of each chunk's request
  int req_end[SCHED_CHUNKS];          // one past the request's last token
  int gbase[SCHED_CHUNKS];            // global position of token t is t + gbase
  unsigned first[SCHED_CHUNKS / 32];  // bit c: chunk c opens its request
};

constexpr int ROPE_MAX_HALF = 64;
struct RopeRow {
  float2* tab;     // [token][half] (cos, sin), or null
  int half;        // d_head / 2 (1 without a table)
  // theta^(-2i / d_head) for i < half, in fp64 (formed on the host: one
  // power per frequency instead of one per table entry)
  double inv_freq[ROPE_MAX_HALF];
};

__global__ __launch_bounds__(256) void schedule_kernel(SchedBatch sb, int* __restrict__ lo,
                                                       int* __restrict__ hi,
                                                       int* __restrict__ pos,
                                                       int* __restrict__ gpos,
                                                       int* __restrict__ flags, RopeRow rr) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int t = sb.offs[0] + (int)(idx / rr.half), i = (int)(idx % rr.half);
  if (t >= sb.offs[sb.count]) return;
  // largest c with offs[c] <= t (skips empty chunks)
  int a = 0, b = sb.count;
  while (b - a > 1) {
    const int mid = (a + b) >> 1;
    if (sb.offs[mid] <= t) a = mid; else b = mid;
  }
  int l = sb.req_start[a], h = sb.offs[a + 1];      // block-causal: c(j) <= c(i)
  if (sb.mask == 1) h = t + 1;                      // token-causal: j <= i
  else if (sb.mask == 2) h = sb.req_end[a];         // bidirectional
  else if (sb.mask == 3) l = sb.offs[a];            // block-diagonal: c(j) == c(i)
  const int p = t - sb.req_start[a];
  if (i == 0) {
    lo[t] = l;
    hi[t] = h;
    pos[t] = p;
    if (gpos) gpos[t] = t + sb.gbase[a];
    if (flags) flags[t] = (sb.first[a >> 5] >> (a & 31)) & 1;
  }
  // (cos, sin)(p * theta^(-2i / d_head)), angle and cosines in fp64
  if (rr.tab) {
    const double ang = (double)p * rr.inv_freq[i];
    rr.tab[(int64_t)t * rr.half + i] = make_float2((float)cos(ang), (float)sin(ang));
  }
}

hipError_t chunk_schedule(const int32_t* off, int32_t n_chunks, const int32_t* req,
                          int32_t n_req, int mask, const int32_t* pos_offset, int* lo, int* hi,
                          int* pos, int* gpos, int* flags, hipStream_t s, float2* rope,
                          int d_head, double theta) {
  RopeRow rr{};
  rr.tab = rope;
  rr.half = rope ? d_head / 2 : 1;
  if (rope && (rr.half < 1 || rr.half > ROPE_MAX_HALF)) return hipErrorInvalidValue;
  if (rope)
    for (int i = 0; i < rr.half; ++i)
      rr.inv_freq[i] = std::pow(theta, -2.0 * (double)i / (double)d_head);
  std::vector<int> rs(n_chunks), re(n_chunks), gb(n_chunks), first(n_chunks);
  const int nr = req ? n_req : 1;
  for (int r = 0; r < nr; ++r) {
    const int c0 = req ? req[r] : 0, c1 = req ? req[r + 1] : n_chunks;
    for (int c = c0; c < c1; ++c) {
      rs[c] = off[c0];
      re[c] = off[c1];
      gb[c] = (pos_offset ? pos_offset[r] : 0) - off[c0];
      first[c] = c == c0;
    }
  }
  for (int c0 = 0; c0 < n_chunks; c0 += SCHED_CHUNKS) {
    SchedBatch sb;
    sb.count = std::min(SCHED_CHUNKS, n_chunks - c0);
    sb.mask = mask;
    for (int i = 0; i <= sb.count; ++i) sb.offs[i] = off[c0 + i];
    for (int i = 0; i < SCHED_CHUNKS / 32; ++i) sb.first[i] = 0;
    for (int i = 0; i < sb.count; ++i) {
      sb.req_start[i] = rs[c0 + i];
      sb.req_end[i] = re[c0 + i];
      sb.gbase[i] = gb[c0 + i];
      sb.first[i >> 5] |= (unsigned)first[c0 + i] << (i & 31);
    }
    const int ntok = sb.offs[sb.count] - sb.offs[0];
    if (ntok == 0) continue;
    const int64_t nthr = (int64_t)ntok * rr.half;
    CR_LAUNCH(schedule_kernel, dim3((unsigned)((nthr + 255) / 256)), dim3(256), 0, s, sb, lo, hi,
              pos, gpos, flags, rr);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// ----------------------------------------------------- paged block table
constexpr int TABLE_BATCH = 512;
struct TableBatch {
  int count;
  int v[TABLE_BATCH];
};

__global__ __launch_bounds__(256) void table_kernel(TableBatch tb, int* __restrict__ dst) {
  for (int i = threadIdx.x; i < tb.count; i += 256) dst[i] = tb.v[i];
}

hipError_t copy_table(const int32_t* host, int n, int* dev, hipStream_t s) {
  for (int i0 = 0; i0 < n; i0 += TABLE_BATCH) {
    TableBatch tb;
    tb.count = std::min(TABLE_BATCH, n - i0);
    for (int i = 0; i < tb.count; ++i) tb.v[i] = host[i0 + i];
    CR_LAUNCH(table_kernel, dim3(1), dim3(256), 0, s, tb, dev + i0);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// ------------------------------------------------- target-model key rotation
// tab[t][i] = scale * (cos, sin)(gpos[t] * f_i), angles and cosines in fp64.
__global__ __launch_bounds__(256) void key_rope_table_kernel(float2* __restrict__ tab,
                                                             const int* __restrict__ gpos, int N,
                                                             KeyRope kr) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)N * kr.half) return;
  const int t = (int)(idx / kr.half), i = (int)(idx % kr.half);
  const double ang = (double)gpos[t] * kr.f[i];
  tab[idx] = make_float2((float)(kr.scale * cos(ang)), (float)(kr.scale * sin(ang)));
}

hipError_t key_rope_table(float2* tab, const int* gpos, int N, const KeyRope& kr, hipStream_t s) {
  const int64_t n = (int64_t)N * kr.half;
  if (n <= 0) return hipSuccess;
  CR_LAUNCH(key_rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, tab, gpos,
            N, kr);
  return hipGetLastError();
}

// One thread rotates 8 rotate-half pairs (i .. i+7, i+half .. i+half+7) of
// one key head of one token, with the (scaled) table of its position:
// forward  k1' = c k1 - s k2,  k2' = c k2 + s k1;
// inverse  k1' = (c k1 + s k2) / scale^2,  k2' = (c k2 - s k1) / scale^2.
template <typename T>
__global__ __launch_bounds__(256) void rotate_keys_kernel(T* __restrict__ kv, KvStrides ks,
                                                          int n_layers, int N,
                                                          const float2* __restrict__ tab,
                                                          int inverse, float inv_scale2) {
  const int half = ks.head_dim / 2, per_head = half / 8;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t per_tok = (int64_t)n_layers * ks.n_kv_heads * per_head;
  if (idx >= (int64_t)N * per_tok) return;
  const int t = (int)(idx / per_tok);
  int rem = (int)(idx % per_tok);
  const int seg8 = rem % per_head;
  rem /= per_head;
  const int h = rem % ks.n_kv_heads, l = rem / ks.n_kv_heads;
  const int i0 = seg8 * 8;
  T* p1 = kv + (int64_t)l * ks.layer + ks.tok(t) + (int64_t)h * ks.head + i0;
  T* p2 = p1 + half;
  Vec8<T> a, b;
  a.load(p1);
  b.load(p2);
  const float4* cs = reinterpret_cast<const float4*>(tab + (int64_t)t * half + i0);
  float x1[8], x2[8], y1[8], y2[8];
  a.to_float(x1);
  b.to_float(x2);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float4 q = cs[e];   // (cos, sin) of pairs 2e and 2e+1
    const float c[2] = {q.x, q.z}, sn[2] = {q.y, q.w};
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int k = 2 * e + u;
      if (inverse) {
        y1[k] = (c[u] * x1[k] + sn[u] * x2[k]) * inv_scale2;
        y2[k] = (c[u] * x2[k] - sn[u] * x1[k]) * inv_scale2;
      } else {
        y1[k] = c[u] * x1[k] - sn[u] * x2[k];
        y2[k] = c[u] * x2[k] + sn[u] * x1[k];
      }
    }
  }
  a.from_float(y1);
  b.from_float(y2);
  a.store(p1);
  b.store(p2);
}

template <typename T>
hipError_t rotate_keys(T* kv, KvStrides ks, int n_layers, int N, const float2* tab, bool inverse,
                       float scale, hipStream_t s) {
  const int64_t n = (int64_t)N * n_layers * ks.n_kv_heads * (ks.head_dim / 16);
  if (n <= 0) return hipSuccess;
  CR_LAUNCH((rotate_keys_kernel<T>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, kv, ks,
            n_layers, N, tab, inverse ? 1 : 0, 1.0f / (scale * scale));
  return hipGetLastError();
}
template hipError_t rotate_keys<bf16>(bf16*, KvStrides, int, int, const float2*, bool, float,
                                      hipStream_t);
template hipError_t rotate_keys<float>(float*, KvStrides, int, int, const float2*, bool, float,
                                       hipStream_t);

// ------------------------------------------------------- weight preparation
// Bias of composed affine maps: out[n] = add[n] (+ add2[n]) + sum_k v[k] W[k][n].
template <typename T>
__global__ __launch_bounds__(256) void compose_bias_kernel(const T* __restrict__ v,
                                                           const T* __restrict__ W, int64_t ldw,
                                                           const T* __restrict__ add,
                                                           const T* __restrict__ add2,
                                                           float* __restrict__ out, int K, int N) {
  const int n = blockIdx.x * 256 + threadIdx.x;
  if (n >= N) return;
  float acc = to_f32(add[n]);
  if (add2) acc += to_f32(add2[n]);
  for (int k = 0; k < K; ++k) acc = fmaf(to_f32(v[k]), to_f32(W[(int64_t)k * ldw + n]), acc);
  out[n] = acc;
}

template <typename T>
hipError_t compose_bias(const T* v, const T* W, int64_t ldw, const T* add, const T* add2,
                        float* out, int K, int N, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  CR_LAUNCH((compose_bias_kernel<T>), dim3((N + 255) / 256), dim3(256), 0, s, v, W, ldw, add, add2,
            out, K, N);
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void transpose_into_kernel(const T* __restrict__ src,
                                                             const T* __restrict__ src2,
                                                             T* __restrict__ dst, int64_t ldd,
                                                             int R, int C) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)R * C) return;
  const int c = (int)(idx / R), r = (int)(idx % R);
  float v = to_f32(src[(int64_t)r * C + c]);
  if (src2) v += to_f32(src2[(int64_t)r * C + c]);
  dst[(int64_t)c * ldd + r] = from_f32<T>(v);
}

template <typename T>
hipError_t transpose_into(const T* src, const T* src2, T* dst, int64_t ldd, int R, int C,
                          hipStream_t s) {
  const int64_t n = (int64_t)R * C;
  if (n <= 0) return hipSuccess;
  CR_LAUNCH((transpose_into_kernel<T>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src,
            src2, dst, ldd, R, C);
  return hipGetLastError();
}

template <typename Tin, typename Tout>
__global__ __launch_bounds__(256) void transpose_convert_kernel(const Tin* __restrict__ src,
                                                                Tout* __restrict__ dst, int R,
                                                                int C, int Cp, int64_t ld_dst,
                                                                const float* __restrict__ div) {
  const int b = blockIdx.z;
  const int64_t n = (int64_t)Cp * ld_dst;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= n) return;
  const int c = (int)(idx / ld_dst), r = (int)(idx % ld_dst);
  float v = 0.f;
  if (c < C && r < R) {
    v = to_f32(src[(int64_t)b * R * C + (int64_t)r * C + c]);
    if (div) v = v / div[(int64_t)b * R + r];
  }
  dst[(int64_t)b * n + idx] = from_f32<Tout>(v);
}

template <typename Tin, typename Tout>
hipError_t transpose_convert(const Tin* src, Tout* dst, int batch, int R, int C, int Cp,
                             int64_t ld_dst, const float* div, hipStream_t s) {
  const int64_t n = (int64_t)Cp * ld_dst;
  if (n <= 0 || batch <= 0) return hipSuccess;
  dim3 grid((unsigned)((n + 255) / 256), 1, batch);
  CR_LAUNCH((transpose_convert_kernel<Tin, Tout>), grid, dim3(256), 0, s, src, dst, R, C,
                     Cp, ld_dst, div);
  return hipGetLastError();
}

template <typename Tin>
__global__ __launch_bounds__(256) void convert_f32_kernel(const Tin* __restrict__ src,
                                                          float* __restrict__ dst, int64_t n,
                                                          int64_t n_pad, int64_t sb, int64_t db) {
  const int b = blockIdx.z;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n_pad) return;
  dst[b * db + i] = i < n ? to_f32(src[b * sb + i]) : 0.f;
}

template <typename Tin>
hipError_t convert_f32(const Tin* src, float* dst, int64_t n, int64_t n_pad, int batch,
                       int64_t sb, int64_t db, hipStream_t s) {
  if (n_pad <= 0 || batch <= 0) return hipSuccess;
  dim3 grid((unsigned)((n_pad + 255) / 256), 1, batch);
  CR_LAUNCH((convert_f32_kernel<Tin>), grid, dim3(256), 0, s, src, dst, n, n_pad, sb, db);
  return hipGetLastError();
}

#define CR_INST(T)                                                                               \
  template hipError_t layernorm<T>(const T*, int64_t, T*, int64_t, const float*, const float*,  \
                                   int, int, float, hipStream_t);                               \
  template hipError_t compress_segments<T>(const T*, KvStrides, int, const T*, const float*, T*, \
                                           int64_t, int, int, hipStream_t);                     \
  template hipError_t transpose_convert<T, T>(const T*, T*, int, int, int, int, int64_t,        \
                                              const float*, hipStream_t);                       \
  template hipError_t convert_f32<T>(const T*, float*, int64_t, int64_t, int, int64_t, int64_t, \
                                     hipStream_t);                                              \
  template hipError_t compose_bias<T>(const T*, const T*, int64_t, const T*, const T*, float*,  \
                                      int, int, hipStream_t);                                   \
  template hipError_t transpose_into<T>(const T*, const T*, T*, int64_t, int, int, hipStream_t);
CR_INST(bf16)
CR_INST(float)
#undef CR_INST

}  // namespace cr
