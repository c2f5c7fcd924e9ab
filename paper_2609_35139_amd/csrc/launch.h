// Host-side launchers of the CacheRepair kernels (internal to the library).
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace cr {

// Profiler events of the stage being enqueued (both null when profiling is
// off).  They are attached to the kernel dispatches themselves, so the pair
// brackets the execution of the stage's kernels on the GPU, not the enqueue:
// the first dispatch of the stage takes the start event, every dispatch the
// stop event.  Thread-local, set around each stage by the library's profiler.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents& launch_events();

#define CR_LAUNCH(KERNEL, GRID, BLOCK, SHMEM, STREAM, ...)                                 \
  do {                                                                                  \
    ::cr::LaunchEvents& le_ = ::cr::launch_events();                                     \
    hipExtLaunchKernelGGL(KERNEL, GRID, BLOCK, SHMEM, STREAM, le_.start, le_.stop, 0,    \
                          __VA_ARGS__);                                                 \
    le_.start = nullptr;                                                                \
  } while (0)

// Cache layout as seen by the kernels (elements).  Strided: token t at
// t*token.  Paged (blocks != null): token t in block blocks[t >> block_shift]
// at row t & (2^block_shift - 1), i.e. blocks[..]*block + row*token.
struct KvStrides {
  int64_t layer, kv, token, head;
  int n_kv_heads, head_dim;
  const int* blocks = nullptr;
  int block_shift = 0;
  int64_t block = 0;
  __device__ __forceinline__ int64_t tok(int t) const {
    if (blocks)
      return (int64_t)blocks[t >> block_shift] * block + (int64_t)(t & ((1 << block_shift) - 1)) * token;
    return (int64_t)t * token;
  }
};

// ---- block table of a paged cache copied from host to device memory
// (passed by value in batches; no host-side staging buffer).
hipError_t copy_table(const int32_t* host, int n, int* dev, hipStream_t s);

// ---- GEMM: C[M][N] = A[M][K] * B[N][K]^T, fp32 accumulation, K % 64 == 0.
// Bias / GELU / residual epilogue: out = (resid +) act(acc + bias) (+ resid2).
template <typename T>
hipError_t gemm_bias(const T* A, int64_t lda, const T* B, int64_t ldb, int M, int N, int K,
                     T* out, int64_t ldo, const float* bias, const T* resid, int64_t ldr,
                     bool gelu, hipStream_t s, const T* resid2 = nullptr, int64_t ldr2 = 0);

// The same with A split along K: C = [A | A2] B^T + bias (+ resid), A
// supplying columns [0, K1) and A2 columns [K1, K); K1 % 64 == 0.
template <typename T>
hipError_t gemm_bias_split(const T* A, int64_t lda, int K1, const T* A2, int64_t lda2, const T* B,
                           int64_t ldb, int M, int N, int K, T* out, int64_t ldo,
                           const float* bias, const T* resid, int64_t ldr, hipStream_t s);

// QKV projection with the repair backbone's RoPE on Q and K (rotate-half
// pairs, table rope[token][d_head/2] of (cos, sin)); Q is written scaled by
// log2(e)/sqrt(d_head); K rows and V^T columns are written up to n_pad
// (finite padding); V is written transposed, vt[head][d][n_pad].
template <typename T>
hipError_t gemm_qkv(const T* A, int64_t lda, const T* B, int M, int K, int d_b, int d_head,
                    T* q, T* k, T* vt, int64_t n_pad, const float* bias, const float2* rope,
                    hipStream_t s);

// KV residual head fused with the output add into the strided cache, for
// coordinates j in [0, D_KV) of the selected components:
//   out[t, j] = (residual ? kv[t, j] : 0) + sigma[j] * (acc[t, j] + bias[j]).
// mode: EXPAND_RESIDUAL | EXPAND_K | EXPAND_V.  keep (may be null): tokens
// with keep[t] != 0 keep their stale values.  With key_rope (may be null,
// table [M][head_dim/2] of scaled (cos, sin), head_dim <= 128) every key head
// of every token is then rotated by its row of the table, whether or not it
// received the output.  out is kv itself (kv_out null: in place, unselected
// coordinates untouched) or kv_out in layout ks_out (every coordinate of
// tokens [0, M) written; kv only read).
enum { EXPAND_RESIDUAL = 1, EXPAND_K = 2, EXPAND_V = 4 };
template <typename T>
hipError_t gemm_expand(const T* A, int64_t lda, const T* B, int M, int N, int K, T* kv,
                       KvStrides ks, const float* bias, const float* sigma, int mode,
                       const int* keep, const float2* key_rope, T* kv_out, KvStrides ks_out,
                       hipStream_t s);

// ---- flash attention over per-row key intervals [lo, hi); q pre-scaled by
// log2(e)/sqrt(d_head); k and vt padded to n_pad >= roundup(N, 64) keys.
// lo and hi must not decrease with the row (chunk_schedule's intervals, for
// every topology, satisfy this): the kernel reads a tile's key range from
// its first and last rows.
template <typename T>
hipError_t attention(const T* q, const T* k, const T* vt, T* o, int N, int d_b, int n_heads,
                     int d_head, int64_t n_pad, const int* lo, const int* hi, hipStream_t s);

// ---- row LayerNorm, C % 8 == 0, C <= 2048.
template <typename T>
hipError_t layernorm(const T* x, int64_t ldx, T* y, int64_t ldy, const float* g, const float* b,
                     int M, int C, float eps, hipStream_t s);

// ---- StaleEncoder stage 1: per-segment projections of the scaled cache into
// U[N][ldu] (segment-major columns g*d_seg + j; columns [S*d_seg, ldu) zeroed).
template <typename T>
hipError_t compress_segments(const T* kv, KvStrides ks, int n_layers, const T* wseg,
                             const float* bseg, T* U, int64_t ldu, int d_seg, int N,
                             hipStream_t s);

// ---- chunk schedule: per token the key interval [lo, hi) of the attention
// topology `mask` (values of CR_MASK_*), the position within the request and,
// when the pointers are not null, the global position (position_offset of the
// request + position; pos_offset may be null = 0), the first-chunk flag and
// the RoPE (cos, sin) row of the position: rope[t][i] = (cos, sin)(pos[t] *
// theta^(-2i / d_head)), i < d_head / 2, computed in fp64.
hipError_t chunk_schedule(const int32_t* chunk_offsets, int32_t n_chunks,
                          const int32_t* request_chunks, int32_t n_requests, int mask,
                          const int32_t* pos_offset, int* lo, int* hi, int* pos, int* gpos,
                          int* flags, hipStream_t s, float2* rope = nullptr, int d_head = 0,
                          double theta = 0.0);

// ---- target-model key rotation R_M(p): frequencies of the rotate-half pairs
// (fp64) and the factor applied to cos and sin.
struct KeyRope {
  int half;
  double scale;
  double f[128];
};
// tab[t][i] = scale * (cos, sin)(gpos[t] * f_i), i < half.
hipError_t key_rope_table(float2* tab, const int* gpos, int N, const KeyRope& kr, hipStream_t s);
// Rotates every key head of tokens [0, N) in place by the table (inverse:
// by the inverse rotation, dividing by scale^2 as well).
template <typename T>
hipError_t rotate_keys(T* kv, KvStrides ks, int n_layers, int N, const float2* tab, bool inverse,
                       float scale, hipStream_t s);

// ---- weight preparation
// out[n] = add[n] (+ add2[n]) + sum_k v[k] * W[k][n] (W row-major [K][ldw]),
// in fp32; K may be 0.
template <typename T>
hipError_t compose_bias(const T* v, const T* W, int64_t ldw, const T* add, const T* add2,
                        float* out, int K, int N, hipStream_t s);
// dst[c][r] = src[r][c] (+ src2[r][c]) for r < R, c < C, summed in fp32 and
// rounded once; dst rows are ldd apart and only their first R entries are
// written (a block inside a wider prepared matrix).
template <typename T>
hipError_t transpose_into(const T* src, const T* src2, T* dst, int64_t ldd, int R, int C,
                          hipStream_t s);
// dst[b][c][r] = src[b][r][c] / div[b][r] for r < R, c < C; zero for
// r in [R, ld_dst) and c in [C, Cp).
template <typename Tin, typename Tout>
hipError_t transpose_convert(const Tin* src, Tout* dst, int batch, int R, int C, int Cp,
                             int64_t ld_dst, const float* div, hipStream_t s);
template <typename Tin>
hipError_t convert_f32(const Tin* src, float* dst, int64_t n, int64_t n_pad, int batch,
                       int64_t src_bstride, int64_t dst_bstride, hipStream_t s);

}  // namespace cr
