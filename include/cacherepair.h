/*
 * cacherepair.h -- C ABI of the CacheRepair repair forward pass on MI355X.
 *
 * The library computes, for the stale canonical KV cache of a packed batch of
 * retrieval requests, the repaired cache
 *
 *     KV_hat = KV_stale + sigma_delta * z,
 *     z      = KVResidualHead(LN(h^B)),
 *
 * where h^B is the output of B Repair Blocks over the fused stale features
 * and token embeddings (paper Section 4.1, "StaleEncoder and token fusion",
 * "Repair Blocks and stale-feature reinjection", "KV residual output and
 * global RoPE").  cr_repair adds in place in the caller's cache and leaves K
 * canonical; cr_repair_ex can place the repaired keys at their global
 * positions in the same pass, runs the paper's controlled variants
 * (attention topologies, entrance-only features, direct prediction, output
 * choices), reads and writes paged caches through a block table and can
 * write the result into a second cache (out of place).  cr_repair_pipelined
 * overlaps the host-to-device copy of one request with the repair of the
 * previous one.  cr_rotate_keys applies the target's rotary encoding (or its
 * inverse) to a cache's keys.
 *
 * Conventions shared by every entry point:
 *  - Plain C: no C++ or torch types.  All sizes are element counts unless the
 *    name ends in _bytes.
 *  - "device" pointers are HIP device memory on the current device; "host"
 *    pointers are read during the call and not retained.
 *  - stream is a hipStream_t passed as void* (NULL = the null stream).  Calls
 *    that take a stream only enqueue work on it and never synchronise;
 *    completion is observed through the stream.
 *  - Every validation happens before anything is enqueued: on an error return
 *    no device memory has been touched.
 *  - The caller owns every buffer.  No call allocates device memory (the one
 *    static device array, cr_repair_static's workspace, is created when the
 *    library's code is loaded on a device).
 *  - Storage dtype (bf16 or fp32) is a property of the cache layout and applies
 *    to the cache, the token embeddings, the canonical weight blob and all
 *    intermediate activations; accumulation is always fp32.  It is a runtime
 *    field of cr_kv_layout, not a build-time choice: one library holds both
 *    the bf16 path and the fp32 debug path, so one process can compare them,
 *    and no "which dtype was this built for" query exists.
 *  - Weights reach the repair calls as the prepared buffer that
 *    cr_prepare_weights builds once from the canonical blob (matrices
 *    transposed to [out][in], 1/sigma_stale folded in, vectors widened to
 *    fp32, and the token projection composed into the fusion: both are
 *    affine with nothing between them, so [s ; t] W_fuse with
 *    t = e W_tok + b_tok is applied as one product of [s ; e], its weights
 *    W_tok W_fuse_t formed on the device and rounded once to the storage
 *    dtype), so no call converts weights; the canonical blob described by
 *    cr_weights_layout stays the one interchange format.
 *  - No exceptions cross the ABI.  Entry points are reentrant given distinct
 *    workspaces.
 */
#ifndef CACHEREPAIR_H
#define CACHEREPAIR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define CR_API __attribute__((visibility("default")))
#else
#define CR_API
#endif

#define CR_ABI_VERSION 1
#define CR_MAX_NAME 48

typedef int32_t cr_status;
enum {
    CR_OK = 0,
    CR_ERR_NULL = -1,       /* a required pointer is NULL                          */
    CR_ERR_DIMS = -2,       /* repairer or cache dimensions outside what is built  */
    CR_ERR_OFFSETS = -3,    /* chunk_offsets / request_chunks malformed            */
    CR_ERR_LAYOUT = -4,     /* cache strides overlap, are misaligned or negative   */
    CR_ERR_WORKSPACE = -5,  /* workspace / prepared / blob buffer too small or
                               misaligned                                          */
    CR_ERR_DTYPE = -6,      /* unknown storage dtype                               */
    CR_ERR_DEVICE = -7,     /* current device is not gfx950 or cannot be queried   */
    CR_ERR_LAUNCH = -8,     /* a kernel launch failed                              */
    CR_ERR_CAPACITY = -9    /* caller's descriptor table is too small              */
};

enum { CR_DTYPE_BF16 = 0, CR_DTYPE_F32 = 1 };

/*
 * Stale canonical cache layout (paper Section 4.1, "Chunk-cache preparation"
 * and "Coordinate convention"): K with local RoPE removed, V native.
 * Element (layer l, component kv in {0 = K, 1 = V}, token t, head h, dim i)
 * lives at  base + l*stride_layer + kv*stride_kv + t*stride_token
 *                + h*stride_head + i        (elements; the dim stride is 1).
 * The map must be injective (strides non-overlapping for the given extents),
 * every stride a non-negative multiple of 8 elements and the base pointer
 * 16-byte aligned.  head_dim must be a multiple of 32 and at most 256.
 * Coordinate j of the residual maps to (l, kv, h, i) with
 * j = ((l*2 + kv)*n_kv_heads + h)*head_dim + i.
 */
typedef struct {
    int32_t n_layers, n_kv_heads, head_dim;
    int32_t dtype;                 /* CR_DTYPE_BF16 or CR_DTYPE_F32 */
    int64_t stride_layer, stride_kv, stride_token, stride_head;
} cr_kv_layout;

/*
 * Repairer dimensions (paper Section 4.1 and Table tab:repair-scales).
 * d_model: width E of the frozen token embedding; d_seg: per-segment
 * projection width (1..32); d_c: width of the compressed stale features s;
 * d_b: repair width; n_heads: attention heads (d_b / n_heads must be 32 or
 * 64); ffn_mult: MLP expansion ratio; rope_theta: base of the repair
 * backbone's RoPE; ln_eps: LayerNorm epsilon.  d_model and d_c must be
 * multiples of 64 and d_b a multiple of 128.
 */
typedef struct {
    int32_t d_model, d_seg, d_c, d_b, n_blocks, n_heads, ffn_mult;
    float rope_theta, ln_eps;
} cr_dims;

/* One tensor of the canonical weight blob. */
typedef struct {
    char name[CR_MAX_NAME];
    int32_t dtype;                 /* CR_DTYPE_*: storage dtype, or F32 for sigma_* */
    int32_t ndim;
    int64_t shape[4];
    uint64_t offset_bytes;         /* from the blob start, 256-byte aligned */
    uint64_t nbytes;
} cr_tensor_desc;

/* ABI version (CR_ABI_VERSION). */
CR_API int32_t cr_version(void);

/* Static, never-NULL description of a status code. */
CR_API const char* cr_status_string(cr_status status);

/*
 * Canonical weight blob layout: every repairer tensor in blob order
 * (paper Section 4.1; matrices are W[in][out] row-major):
 *   w_seg[S][d_h][d_seg] b_seg[S][d_seg]  w_cmp[S*d_seg][d_c] b_cmp[d_c]
 *   ln_enc_g[d_c] ln_enc_b[d_c]  w_tok[E][d_b] b_tok[d_b]
 *   w_fuse[d_c+d_b][d_b] b_fuse[d_b]
 *   per block b: blk<b>.{w_inj[d_c][d_b] b_inj ln1_g ln1_b w_qkv[d_b][3d_b]
 *                b_qkv w_o[d_b][d_b] b_o ln2_g ln2_b w_ff1[d_b][r*d_b] b_ff1
 *                w_ff2[r*d_b][d_b] b_ff2}
 *   ln_f_g[d_b] ln_f_b[d_b]  w_out[d_b][D_KV] b_out[D_KV]
 *   sigma_stale[D_KV] sigma_delta[D_KV]        (always fp32)
 * w_qkv columns are Q | K | V, each head-major (column h*d_head + i).
 * entries: host array of max_entries descriptors (may be NULL to query only
 * the count); n_entries and total_bytes: host outputs.
 * Errors: CR_ERR_NULL, CR_ERR_DIMS, CR_ERR_DTYPE, CR_ERR_CAPACITY.
 */
CR_API cr_status cr_weights_layout(const cr_dims* dims, const cr_kv_layout* layout,
                            cr_tensor_desc* entries, int32_t max_entries,
                            int32_t* n_entries, uint64_t* total_bytes);

/* Size of the prepared (device-optimised) weight buffer. */
CR_API cr_status cr_prepared_bytes(const cr_dims* dims, const cr_kv_layout* layout,
                            uint64_t* bytes);

/*
 * One-time load step: converts the canonical blob (device, as described by
 * cr_weights_layout) into the prepared buffer (device, cr_prepared_bytes):
 * matrices transposed to [out][in], 1/sigma_stale folded into w_seg, vectors
 * widened to fp32.  Exact in real arithmetic; the folded w_seg is rounded
 * once to the storage dtype.  Both buffers 256-byte aligned.
 */
CR_API cr_status cr_prepare_weights(const cr_dims* dims, const cr_kv_layout* layout,
                             const void* blob, uint64_t blob_bytes,
                             void* prepared, uint64_t prepared_bytes, void* stream);

/* Device workspace needed by cr_repair for a packed batch of n_tokens tokens. */
CR_API cr_status cr_workspace_bytes(const cr_dims* dims, const cr_kv_layout* layout,
                             int64_t n_tokens, uint64_t* bytes);

/*
 * Chunk schedule of the block-causal mask A_ij = 1[c(j) <= c(i)] (paper
 * Section 4.1, Repair Blocks), restricted to tokens of the same request.
 * For every token t it writes, to the device array rows[3*N] (N =
 * chunk_offsets[n_chunks]):
 *   rows[t]       = lo(t): first token of t's request,
 *   rows[N + t]   = hi(t): one past the last token of t's chunk,
 *   rows[2N + t]  = p_t:   0-based position of t within its request,
 * so that t attends exactly to keys j with lo(t) <= j < hi(t).
 * chunk_offsets: host, n_chunks+1 token offsets (0 = first, non-decreasing,
 * empty chunks allowed).  request_chunks: host, n_requests+1 chunk offsets
 * (first 0, last n_chunks, non-decreasing), or NULL for one request.
 * cr_repair uses the same kernel internally.
 */
CR_API cr_status cr_chunk_schedule(const int32_t* chunk_offsets, int32_t n_chunks,
                            const int32_t* request_chunks, int32_t n_requests,
                            int32_t* rows, void* stream);

/*
 * The repair forward pass, in place.
 *  kv:            device, IN/OUT, stale canonical cache in `layout`; only the
 *                 coordinates of tokens [0, N) are read and written.
 *  chunk_offsets, n_chunks, request_chunks, n_requests: as cr_chunk_schedule;
 *                 N = chunk_offsets[n_chunks] tokens, packed request by request.
 *  token_embeds:  device, [N][d_model] row-major, storage dtype: the frozen
 *                 target embeddings E_M(x_t), already gathered.
 *  prepared:      device, output of cr_prepare_weights for the same dims and
 *                 layout.
 *  workspace:     device scratch of at least cr_workspace_bytes(N) bytes,
 *                 256-byte aligned; must not alias kv, token_embeds or
 *                 prepared.  Contents are undefined after the call.
 * N == 0 returns CR_OK with nothing enqueued.
 * Errors: CR_ERR_NULL, CR_ERR_DIMS, CR_ERR_OFFSETS, CR_ERR_LAYOUT,
 * CR_ERR_WORKSPACE, CR_ERR_DTYPE, CR_ERR_DEVICE (before any enqueue);
 * CR_ERR_LAUNCH if a launch fails (earlier launches may have run).
 */
CR_API cr_status cr_repair(void* kv, const cr_kv_layout* layout,
                    const int32_t* chunk_offsets, int32_t n_chunks,
                    const int32_t* request_chunks, int32_t n_requests,
                    const void* token_embeds, const cr_dims* dims,
                    const void* prepared, uint64_t prepared_bytes,
                    void* workspace, uint64_t workspace_bytes, void* stream);

/*
 * Variants of the repair forward pass and global placement of the keys.
 *
 * Attention topology of the repair blocks (paper appendix "Attention
 * Topology and Within-Chunk Context"; every topology only allows keys of the
 * query's own request):
 *   CR_MASK_BLOCK_CAUSAL    A0, the method: c(j) <= c(i)
 *   CR_MASK_TOKEN_CAUSAL    A1: j <= i
 *   CR_MASK_BIDIRECTIONAL   A2: every token of the request
 *   CR_MASK_BLOCK_DIAGONAL  A3: c(j) == c(i)
 * Output components that receive the network's correction (Table
 * tab:repair-components; the network runs in full in every case):
 *   CR_APPLY_KV (the method), CR_APPLY_K, CR_APPLY_V.
 */
enum {
    CR_MASK_BLOCK_CAUSAL = 0,
    CR_MASK_TOKEN_CAUSAL = 1,
    CR_MASK_BIDIRECTIONAL = 2,
    CR_MASK_BLOCK_DIAGONAL = 3
};
enum { CR_APPLY_KV = 0, CR_APPLY_K = 1, CR_APPLY_V = 2 };

/*
 * The target model's rotary encoding R_M (paper Section 4.1, "Chunk-cache
 * preparation" and "KV residual output and global RoPE").  Every K head is
 * rotated in rotate-half pairs (i, i + head_dim/2) by the angle p * f_i, and
 * both rotated values are multiplied by scale:
 *   k'_i          = scale * ( k_i cos(p f_i) - k_{i+d/2} sin(p f_i) )
 *   k'_{i+d/2}    = scale * ( k_{i+d/2} cos(p f_i) + k_i sin(p f_i) )
 * f_i = theta^(-2i/head_dim) when inv_freq is NULL; otherwise inv_freq is a
 * host array of head_dim/2 frequencies (radians per position), which covers
 * the models' frequency-scaling rules.  scale is 1 for plain RoPE.  Angles
 * and their cosines are evaluated in fp64.
 */
typedef struct {
    double theta;              /* > 0; used when inv_freq is NULL           */
    const float* inv_freq;     /* host, head_dim/2 entries, or NULL         */
    float scale;               /* > 0                                       */
} cr_rope;

/*
 * Options of cr_repair_ex.  cr_default_options gives the method:
 * block-causal mask, per-block reinjection, residual output on K and V,
 * canonical keys.
 *  mask:             CR_MASK_*.
 *  reinject:         1 = every block adds P_b(s) + b_b (the method); 0 =
 *                    variant A4, stale features enter only through token
 *                    fusion (the blob keeps its w_inj/b_inj entries, unused).
 *  residual:         1 = KV_hat = KV_stale + sigma_delta * z (the method);
 *                    0 = variant A5, direct prediction with zero output
 *                    offset, KV_hat = sigma_delta * z.
 *  apply:            CR_APPLY_*: components that receive the output; the
 *                    others keep their stale values.
 *  keep_first_chunk: 1 = the tokens of the first chunk of every request
 *                    (chunk index request_chunks[r]) keep their stale values.
 *  global_rope:      NULL = keys stay canonical (the method as cr_repair
 *                    computes it); otherwise, after the output add, every key
 *                    of token t is placed at its global request position,
 *                    K_hat_t = R_M(p_t) K_hat_t^c, fused into the output add.
 *                    Requires head_dim <= 128.
 *  position_offset:  host, n_requests entries (NULL = all 0): global position
 *                    of the first document token of each request (e.g. the
 *                    length of a cached preamble); p_t = position_offset[r] +
 *                    position of t within its request.  Each p_t must be
 *                    non-negative and below 2^31 - 1.
 *  pages:            NULL, or a paged cache layout (cr_kv_pages).
 *  kv_out, layout_out, pages_out: when kv_out is not NULL the repaired cache
 *                    is written there (device, layout_out with the same
 *                    n_layers, n_kv_heads, head_dim and dtype as layout,
 *                    optionally paged) and kv is only read: the write into
 *                    the serving cache is fused into the output add.  Every
 *                    coordinate of tokens [0, N) of kv_out is written; kv_out
 *                    must not overlap kv, token_embeds or the workspace.
 */
/*
 * Paged cache (the block-table layout of paged serving caches; the paper's
 * baselines inject repaired prefixes into a paged cache of 16-token blocks,
 * appendix "Cached-prefix execution", and time that write separately, Table
 * tab:repair-latency-components, "KV write").  With pages, the repair reads
 * and writes the blocks in place and no separate write is needed.
 * Token t of the batch lives in block block_table[t / block_size], row
 * t % block_size, so element (l, kv, t, h, i) is at
 *   base + l*stride_layer + kv*stride_kv + block_table[t / block_size]*stride_block
 *        + (t % block_size)*stride_token + h*stride_head + i
 * (stride_* other than stride_block from cr_kv_layout).
 *  block_size:   tokens per block, a power of two, 1..1024.
 *  n_blocks:     blocks the cache holds (block ids lie in [0, n_blocks)).
 *  stride_block: elements between consecutive blocks (a multiple of 8).
 *  block_table:  host, ceil(N / block_size) distinct block ids.
 * The strides must be injective over (layer, kv, block, row, head, dim) for
 * n_blocks blocks; otherwise CR_ERR_LAYOUT.  A bad table (id out of range or
 * repeated) gives CR_ERR_LAYOUT before anything is enqueued.
 */
typedef struct {
    int32_t block_size;
    int32_t n_blocks;
    int64_t stride_block;
    const int32_t* block_table;
} cr_kv_pages;

typedef struct {
    int32_t mask;
    int32_t reinject;
    int32_t residual;
    int32_t apply;
    int32_t keep_first_chunk;
    const cr_rope* global_rope;
    const int32_t* position_offset;
    const cr_kv_pages* pages;    /* NULL = the strided layout of cr_kv_layout */
    void* kv_out;                    /* NULL = repair in place                 */
    const cr_kv_layout* layout_out;  /* layout of kv_out (required with it)    */
    const cr_kv_pages* pages_out;    /* NULL = strided layout_out              */
} cr_options;

/* Fills opt with the method's options. */
CR_API void cr_default_options(cr_options* opt);

/*
 * cr_repair with options (see cr_options); cr_repair(...) is
 * cr_repair_ex(..., &defaults).  Same buffers, errors and asynchrony as
 * cr_repair; options outside their ranges, a NULL/invalid global_rope field
 * or head_dim > 128 with global_rope give CR_ERR_DIMS, offsets that put a
 * position outside [0, 2^31 - 1) give CR_ERR_OFFSETS.
 */
CR_API cr_status cr_repair_ex(void* kv, const cr_kv_layout* layout,
                       const int32_t* chunk_offsets, int32_t n_chunks,
                       const int32_t* request_chunks, int32_t n_requests,
                       const void* token_embeds, const cr_dims* dims,
                       const void* prepared, uint64_t prepared_bytes,
                       void* workspace, uint64_t workspace_bytes, void* stream,
                       const cr_options* options);

/*
 * Rotates every key of tokens [0, N) of a cache in place by R_M(p_t)
 * (inverse = 0) or R_M(p_t)^-1 (inverse = 1), with p_t as in cr_options
 * (position within the request plus position_offset[r]); V is not touched.
 * inverse = 1 with one chunk per request turns independently prefilled
 * chunk caches into canonical coordinates (paper Section 4.1, "Chunk-cache
 * preparation"); inverse = 0 places canonical keys at global positions.
 * kv, layout, chunk_offsets, n_chunks, request_chunks, n_requests: as
 * cr_repair; pages: NULL or a paged layout (cr_kv_pages).  workspace: device,
 * at least cr_rotate_workspace_bytes bytes, 256-byte aligned.  Requires
 * head_dim <= 256.  Errors as cr_repair_ex.
 */
CR_API cr_status cr_rotate_workspace_bytes(const cr_kv_layout* layout, int64_t n_tokens,
                                    uint64_t* bytes);
CR_API cr_status cr_rotate_keys(void* kv, const cr_kv_layout* layout,
                         const int32_t* chunk_offsets, int32_t n_chunks,
                         const int32_t* request_chunks, int32_t n_requests,
                         const cr_rope* rope, const int32_t* position_offset,
                         int32_t inverse, const cr_kv_pages* pages,
                         void* workspace, uint64_t workspace_bytes, void* stream);

/*
 * Pipelined repair of a sequence of requests whose stale caches sit in
 * pinned host memory (the transfer is the largest TTFT component for the
 * larger targets, Table tab:repair-latency-components, "H2D"; overlapping it
 * with repair across requests is the paper's stated next step).  Request i
 * is copied host -> device into staging slot i % 2 on copy_stream while
 * request i - 1 is repaired on compute_stream from the other slot, straight
 * into its destination cache (out of place, optionally paged).  Events of
 * the handle order the two streams; a slot is refilled only after the
 * repair that read it has finished, also across calls on one handle.  The
 * host buffers must stay valid until copy_stream has passed the copies;
 * each destination is complete once compute_stream has passed the call.
 *
 * cr_pipeline_create / cr_pipeline_destroy: the handle holds four HIP events
 * (created here, never inside cr_repair_pipelined).  A handle serves one
 * cr_repair_pipelined call at a time.
 * cr_pipeline_staging_bytes: device staging for two slots of max_tokens
 * tokens (cache [L][2][n][H][d_h] and embeddings [n][d_model]).
 */
typedef struct {
    const void* kv_host;             /* pinned host, stale canonical cache, layer-major
                                        [L][2][n][H][d_h], n = chunk_offsets[n_chunks] */
    const void* embeds_host;         /* pinned host, [n][d_model]                    */
    const int32_t* chunk_offsets;    /* host, n_chunks+1 token offsets (one request) */
    int32_t n_chunks;
    int32_t position_offset;         /* global position of the first token (with
                                        options->global_rope)                       */
    void* kv_out;                    /* device destination cache                     */
    const cr_kv_layout* layout_out;  /* its layout (n = its token extent)            */
    const cr_kv_pages* pages_out;    /* NULL = strided                               */
} cr_pipeline_item;

typedef struct cr_pipeline_s* cr_pipeline;

CR_API cr_status cr_pipeline_create(cr_pipeline* pipeline);
CR_API cr_status cr_pipeline_destroy(cr_pipeline pipeline);
CR_API cr_status cr_pipeline_staging_bytes(const cr_dims* dims, const cr_kv_layout* layout,
                                    int64_t max_tokens, uint64_t* bytes);
/*
 * items: host array of n_items requests, each at most max_tokens tokens.
 * layout: n_layers, n_kv_heads, head_dim and dtype of every request's cache
 * (strides ignored).  staging, workspace: device, cr_pipeline_staging_bytes
 * and cr_workspace_bytes for max_tokens, 256-byte aligned.  options: the
 * variant (its pages, kv_out, layout_out, pages_out and position_offset are
 * ignored: they come from the items), or NULL for the method.
 * copy_stream and compute_stream must be distinct.  Validation of every
 * item happens before anything is enqueued.
 */
CR_API cr_status cr_repair_pipelined(cr_pipeline pipeline, const cr_pipeline_item* items,
                              int32_t n_items, const cr_dims* dims, const cr_kv_layout* layout,
                              const void* prepared, uint64_t prepared_bytes, void* staging,
                              uint64_t staging_bytes, int64_t max_tokens, void* workspace,
                              uint64_t workspace_bytes, const cr_options* options,
                              void* copy_stream, void* compute_stream);

/*
 * Debug view into the workspace after a cr_repair call that has completed:
 * name is "s" (stale features, [N][d_c]), "h" (h^B, [N][d_b]) or "lnf"
 * (LN_f(h^B), [N][d_b]).  Returns the byte offset from the workspace start
 * and the row stride in elements.  These buffers hold the final values of a
 * completed call and are overwritten by the next one.
 */
CR_API cr_status cr_workspace_view(const cr_dims* dims, const cr_kv_layout* layout,
                            int64_t n_tokens, const char* name,
                            uint64_t* offset_bytes, int64_t* row_stride);

/*
 * cr_repair without a caller workspace, for callers that cannot allocate
 * device memory: code under HIP graph capture, serving loops that forbid
 * hipMalloc, harnesses without an allocator.  Same arguments as cr_repair
 * minus the workspace; same kernels and bit-identical results.  The
 * workspace is a device array inside the library of CR_STATIC_SCRATCH_BYTES
 * bytes (128 MiB: enough for a 4,096-token request of a Qwen2.5-3B-shaped
 * cache with a d_b = 1024, 8-block repairer, which needs 118.1 MiB), held by
 * every GPU the library runs on until the process ends.  A call needing more (see
 * cr_workspace_bytes) returns CR_ERR_WORKSPACE before anything is enqueued.
 * The call allocates nothing, on the host or the device.  Every call on one
 * GPU uses that GPU's one array, which keeps the previous call's contents
 * (the repair writes every workspace byte it reads): calls that overlap in
 * time on one GPU (several streams or threads) race, so serialise them,
 * e.g. on one stream.  Errors as cr_repair; CR_ERR_DEVICE also when the
 * array's device address cannot be obtained.
 */
#define CR_STATIC_SCRATCH_BYTES (128ull << 20)
CR_API cr_status cr_repair_static(void* kv, const cr_kv_layout* layout,
                                  const int32_t* chunk_offsets, int32_t n_chunks,
                                  const int32_t* request_chunks, int32_t n_requests,
                                  const void* token_embeds, const cr_dims* dims,
                                  const void* prepared, uint64_t prepared_bytes, void* stream);

/*
 * Per-launch timing (tracing aid, not needed for repair).  While enabled,
 * cr_repair brackets every kernel launch with HIP events recorded on the
 * call's own stream.  cr_profile_enable(max_launches) creates the events
 * (host-side allocation happens here, never inside cr_repair);
 * max_launches = 0 disables profiling and destroys them.  Launches beyond
 * max_launches since the last reset are not timed.  cr_profile_read waits for
 * the recorded events, then fills up to max_stats entries, one per kernel
 * class in first-launch order, and resets the record (also when it returns
 * an error).  A stage whose launch failed is left out of the record: its
 * events were never recorded.  This is process-wide state guarded by a
 * mutex, held while a timed stage is enqueued (so cr_profile_enable waits
 * for it); profile one stream at a time.
 */
typedef struct {
    char name[32];        /* kernel class, e.g. "attention", "gemm_ffn1" */
    int32_t launches;
    double total_ms;
} cr_kernel_stat;

CR_API cr_status cr_profile_enable(int32_t max_launches);
CR_API cr_status cr_profile_read(cr_kernel_stat* stats, int32_t max_stats, int32_t* n_stats);

#ifdef __cplusplus
}
#endif
#endif /* CACHEREPAIR_H */
