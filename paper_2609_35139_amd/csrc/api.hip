// C ABI of the CacheRepair repair forward pass: validation, buffer layouts
// and the kernel sequence of one call.  See include/cacherepair.h.
#include "../../include/cacherepair.h"

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "launch.h"

namespace cr {
LaunchEvents& launch_events() {
  static thread_local LaunchEvents le;
  return le;
}
}  // namespace cr

namespace {

using cr::bf16;
using cr::LaunchEvents;
using cr::launch_events;

constexpr uint64_t ALIGN = 256;
inline uint64_t align_up(uint64_t x, uint64_t a = ALIGN) { return (x + a - 1) / a * a; }
inline int64_t round_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

struct Arena {
  uint64_t off = 0;
  uint64_t take(uint64_t bytes) {
    const uint64_t o = off;
    off = align_up(off + bytes);
    return o;
  }
};

inline size_t esize(int dtype) { return dtype == CR_DTYPE_F32 ? 4 : 2; }

// ------------------------------------------------------------ validation
cr_status check_dtype(const cr_kv_layout* l) {
  return (l->dtype == CR_DTYPE_BF16 || l->dtype == CR_DTYPE_F32) ? CR_OK : CR_ERR_DTYPE;
}

cr_status check_dims(const cr_dims* d, const cr_kv_layout* l) {
  if (!d || !l) return CR_ERR_NULL;
  cr_status st = check_dtype(l);
  if (st != CR_OK) return st;
  if (l->n_layers < 1 || l->n_kv_heads < 1 || l->head_dim < 32 || l->head_dim > 256 ||
      l->head_dim % 32 != 0)
    return CR_ERR_DIMS;
  if ((int64_t)2 * l->n_layers * l->n_kv_heads * l->head_dim > (int64_t)1 << 24) return CR_ERR_DIMS;
  if (d->d_model < 64 || d->d_model % 64 != 0) return CR_ERR_DIMS;
  if (d->d_seg < 1 || d->d_seg > 32) return CR_ERR_DIMS;
  if (d->d_c < 64 || d->d_c % 64 != 0 || d->d_c > 2048) return CR_ERR_DIMS;
  if (d->d_b < 128 || d->d_b % 128 != 0 || d->d_b > 2048) return CR_ERR_DIMS;
  if (d->n_heads < 1 || d->d_b % d->n_heads != 0) return CR_ERR_DIMS;
  const int dh = d->d_b / d->n_heads;
  if (dh != 32 && dh != 64) return CR_ERR_DIMS;
  if (d->n_blocks < 0 || d->n_blocks > 256) return CR_ERR_DIMS;
  if (d->ffn_mult < 1 || d->ffn_mult > 16) return CR_ERR_DIMS;
  if (!(d->rope_theta > 0.f) || !(d->ln_eps >= 0.f)) return CR_ERR_DIMS;
  return CR_OK;
}

// Injective index map over (stride, extent) pairs: with the dims sorted by
// stride, each stride must exceed the largest offset reachable through the
// dims inside it.  The largest offset must also stay below 2^62 elements, so
// that no element offset a kernel forms in int64 can overflow.
struct Dim { int64_t s, e; };
// At most six (stride, extent) pairs: dim, head, token, (block,) K/V, layer.
// Fixed capacity, so validating a call allocates nothing.
struct Dims {
  Dim d[6];
  int n = 0;
  void push_back(Dim x) { d[n++] = x; }
};
cr_status check_injective(Dims dims) {
  std::sort(dims.d, dims.d + dims.n, [](const Dim& a, const Dim& b) { return a.s < b.s; });
  int64_t reach = 0;  // largest offset reachable by the dims visited so far
  for (int i = 0; i < dims.n; ++i) {
    const Dim& x = dims.d[i];
    if (x.s <= reach) return CR_ERR_LAYOUT;
    int64_t span;
    if (__builtin_mul_overflow(x.s, x.e - 1, &span) || __builtin_add_overflow(reach, span, &reach) ||
        reach >= ((int64_t)1 << 62))
      return CR_ERR_LAYOUT;
  }
  return CR_OK;
}

cr_status check_layout(const cr_kv_layout* l, int64_t n_tokens) {
  const int64_t st[4] = {l->stride_layer, l->stride_kv, l->stride_token, l->stride_head};
  const int64_t ext[4] = {l->n_layers, 2, n_tokens, l->n_kv_heads};
  Dims dims;
  dims.push_back({1, l->head_dim});
  for (int i = 0; i < 4; ++i) {
    if (st[i] < 0 || st[i] % 8 != 0) return CR_ERR_LAYOUT;
    if (ext[i] > 1) dims.push_back({st[i], ext[i]});
  }
  if (n_tokens == 0) return CR_OK;  // no element is addressed
  return check_injective(dims);
}

// Injectivity of a paged layout over (layer, kv, block, row, head, dim) and
// validity of the host block table for n_tokens tokens.
cr_status check_pages(const cr_kv_layout* l, const cr_kv_pages* pg, int64_t n_tokens) {
  const int bs = pg->block_size;
  if (bs < 1 || bs > 1024 || (bs & (bs - 1)) || pg->n_blocks < 1) return CR_ERR_LAYOUT;
  if (pg->stride_block < 0 || pg->stride_block % 8) return CR_ERR_LAYOUT;
  const int64_t st[5] = {l->stride_layer, l->stride_kv, pg->stride_block, l->stride_token,
                         l->stride_head};
  const int64_t ext[5] = {l->n_layers, 2, pg->n_blocks, bs, l->n_kv_heads};
  Dims dims;
  dims.push_back({1, l->head_dim});
  for (int i = 0; i < 5; ++i) {
    if (st[i] < 0 || st[i] % 8 != 0) return CR_ERR_LAYOUT;
    if (ext[i] > 1) dims.push_back({st[i], ext[i]});
  }
  const cr_status inj = check_injective(dims);
  if (inj != CR_OK) return inj;
  const int64_t nb = (n_tokens + bs - 1) / bs;
  if (nb == 0) return CR_OK;
  if (!pg->block_table) return CR_ERR_NULL;
  std::vector<int32_t> ids(pg->block_table, pg->block_table + nb);
  for (int32_t b : ids)
    if (b < 0 || b >= pg->n_blocks) return CR_ERR_LAYOUT;
  std::sort(ids.begin(), ids.end());
  if (std::adjacent_find(ids.begin(), ids.end()) != ids.end()) return CR_ERR_LAYOUT;
  return CR_OK;
}

int log2_int(int x) {
  int s = 0;
  while ((1 << s) < x) ++s;
  return s;
}

cr_status check_offsets(const int32_t* off, int32_t n_chunks, const int32_t* req,
                        int32_t n_req) {
  if (!off) return CR_ERR_NULL;
  if (n_chunks < 1) return CR_ERR_OFFSETS;
  if (off[0] != 0) return CR_ERR_OFFSETS;
  for (int i = 0; i < n_chunks; ++i)
    if (off[i + 1] < off[i]) return CR_ERR_OFFSETS;
  if (req) {
    if (n_req < 1 || req[0] != 0 || req[n_req] != n_chunks) return CR_ERR_OFFSETS;
    for (int i = 0; i < n_req; ++i)
      if (req[i + 1] < req[i]) return CR_ERR_OFFSETS;
  }
  return CR_OK;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Target rotary encoding: frequencies in fp64 from theta or the caller's
// table.  Returns CR_ERR_DIMS for a non-finite or non-positive field.
cr_status key_rope_of(const cr_rope* r, int head_dim, cr::KeyRope* kr) {
  if (!r || head_dim / 2 > 128) return CR_ERR_DIMS;
  if (!(r->scale > 0.f) || !std::isfinite(r->scale)) return CR_ERR_DIMS;
  kr->half = head_dim / 2;
  kr->scale = r->scale;
  for (int i = 0; i < kr->half; ++i) {
    double f;
    if (r->inv_freq) {
      f = r->inv_freq[i];
    } else {
      if (!(r->theta > 0.0) || !std::isfinite(r->theta)) return CR_ERR_DIMS;
      f = std::pow(r->theta, -2.0 * i / (double)head_dim);
    }
    if (!std::isfinite(f)) return CR_ERR_DIMS;
    kr->f[i] = f;
  }
  return CR_OK;
}

// Global positions p_t = position_offset[r] + (t - first token of r) must lie
// in [0, 2^31 - 1).
cr_status check_positions(const int32_t* off, int32_t n_chunks, const int32_t* req,
                          int32_t n_req, const int32_t* pos_offset) {
  const int nr = req ? n_req : 1;
  for (int r = 0; r < nr; ++r) {
    const int64_t o = pos_offset ? pos_offset[r] : 0;
    const int64_t len = req ? (int64_t)off[req[r + 1]] - off[req[r]] : off[n_chunks];
    if (o < 0 || o + len >= ((int64_t)1 << 31) - 1) return CR_ERR_OFFSETS;
  }
  return CR_OK;
}

cr_status check_device() {
  static std::atomic<int> ok[64];  // per device: 0 unknown, 1 gfx950, -1 not
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return CR_ERR_DEVICE;
  const int known = dev < 64 ? ok[dev].load(std::memory_order_relaxed) : 0;
  if (known) return known > 0 ? CR_OK : CR_ERR_DEVICE;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return CR_ERR_DEVICE;
  const bool good = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
  if (dev < 64) ok[dev].store(good ? 1 : -1, std::memory_order_relaxed);
  return good ? CR_OK : CR_ERR_DEVICE;
}

// ------------------------------------------------------------- layouts
struct Tensor {
  std::string name;
  int dtype;
  std::vector<int64_t> shape;
  uint64_t off = 0, nbytes = 0;
};

// Canonical blob: every tensor of the repairer in blob order.
std::vector<Tensor> canonical(const cr_dims* d, const cr_kv_layout* l, uint64_t* total) {
  const int T = l->dtype;
  const int64_t S = 2LL * l->n_layers * l->n_kv_heads, dh = l->head_dim, D = S * dh;
  const int64_t dc = d->d_c, db = d->d_b, E = d->d_model, r = d->ffn_mult, ds = d->d_seg;
  std::vector<Tensor> v;
  auto add = [&](const std::string& n, int dt, std::vector<int64_t> sh) { v.push_back({n, dt, sh}); };
  add("w_seg", T, {S, dh, ds}); add("b_seg", T, {S, ds});
  add("w_cmp", T, {S * ds, dc}); add("b_cmp", T, {dc});
  add("ln_enc_g", T, {dc}); add("ln_enc_b", T, {dc});
  add("w_tok", T, {E, db}); add("b_tok", T, {db});
  add("w_fuse", T, {dc + db, db}); add("b_fuse", T, {db});
  for (int b = 0; b < d->n_blocks; ++b) {
    const std::string p = "blk" + std::to_string(b) + ".";
    add(p + "w_inj", T, {dc, db}); add(p + "b_inj", T, {db});
    add(p + "ln1_g", T, {db}); add(p + "ln1_b", T, {db});
    add(p + "w_qkv", T, {db, 3 * db}); add(p + "b_qkv", T, {3 * db});
    add(p + "w_o", T, {db, db}); add(p + "b_o", T, {db});
    add(p + "ln2_g", T, {db}); add(p + "ln2_b", T, {db});
    add(p + "w_ff1", T, {db, r * db}); add(p + "b_ff1", T, {r * db});
    add(p + "w_ff2", T, {r * db, db}); add(p + "b_ff2", T, {db});
  }
  add("ln_f_g", T, {db}); add("ln_f_b", T, {db});
  add("w_out", T, {db, D}); add("b_out", T, {D});
  add("sigma_stale", CR_DTYPE_F32, {D}); add("sigma_delta", CR_DTYPE_F32, {D});
  Arena a;
  for (Tensor& t : v) {
    uint64_t n = 1;
    for (int64_t s : t.shape) n *= (uint64_t)s;
    t.nbytes = n * esize(t.dtype);
    t.off = a.take(t.nbytes);
  }
  *total = a.off;
  return v;
}

struct BlockP {
  uint64_t ln1_g, ln1_b, w_qkv, b_qkv, w_o, b_o, ln2_g, ln2_b, w_ff1, b_ff1, w_ff2, b_ff2,
      b_ff2_rj;
};
// Prepared (device-optimised) weights: matrices [out][in] in the storage
// dtype, vectors fp32.  Each reinjection x_b = h^b + s W_inj_b + b_inj_b
// follows an affine step with nothing in between, so it is folded into that
// step's product: block 0's into the fusion (W_fuse_s + W_inj_0 on the s
// columns), block b's into block b-1's FFN2, whose rows carry d_c more
// columns (W_inj_b, applied to s: K grows from r*d_b to r*d_b + d_c).  The
// entrance-only variant uses the plain fusion matrix and the first r*d_b
// columns of the FFN2 rows.  The blocks' tensors follow one another with the
// same layout, so block b's offsets are block 0's plus b times the block
// stride.
struct Prepared {
  int64_t kc, kc_pad;
  uint64_t w_seg, b_seg, w_cmp, b_cmp, ln_enc_g, ln_enc_b, w_fuse, b_fuse, w_fuse_rj, b_fuse_rj;
  BlockP blk0;
  uint64_t blk_stride;
  uint64_t ln_f_g, ln_f_b, w_out, b_out, sigma_delta;
  uint64_t tmp;   // scratch of the preparation itself
  uint64_t total;
  BlockP blk(int b) const {
    const uint64_t o = (uint64_t)b * blk_stride;
    const BlockP& q = blk0;
    return BlockP{q.ln1_g + o, q.ln1_b + o, q.w_qkv + o, q.b_qkv + o, q.w_o + o, q.b_o + o,
                  q.ln2_g + o, q.ln2_b + o, q.w_ff1 + o, q.b_ff1 + o, q.w_ff2 + o, q.b_ff2 + o,
                  q.b_ff2_rj + o};
  }
};

Prepared prepared_layout(const cr_dims* d, const cr_kv_layout* l) {
  const size_t T = esize(l->dtype), F = 4;
  const int64_t S = 2LL * l->n_layers * l->n_kv_heads, dh = l->head_dim, D = S * dh;
  const int64_t dc = d->d_c, db = d->d_b, E = d->d_model, r = d->ffn_mult;
  Prepared p;
  p.kc = S * d->d_seg;
  p.kc_pad = round_up(p.kc, 64);
  Arena a;
  p.w_seg = a.take(S * 32 * dh * T);
  p.b_seg = a.take(S * 32 * F);
  p.w_cmp = a.take(dc * p.kc_pad * T);
  p.b_cmp = a.take(dc * F); p.ln_enc_g = a.take(dc * F); p.ln_enc_b = a.take(dc * F);
  // the fusion [s ; t] W_fuse with t = e W_tok + b_tok, composed into one
  // map of [s ; e]: [W_fuse_s ; W_tok W_fuse_t], bias b_fuse + b_tok W_fuse_t
  p.w_fuse = a.take(db * (dc + E) * T); p.b_fuse = a.take(db * F);
  p.w_fuse_rj = a.take(db * (dc + E) * T); p.b_fuse_rj = a.take(db * F);   // + block 0's P_0
  const uint64_t first = a.off;
  for (int b = 0; b < d->n_blocks; ++b) {
    BlockP q;
    q.ln1_g = a.take(db * F); q.ln1_b = a.take(db * F);
    q.w_qkv = a.take(3 * db * db * T); q.b_qkv = a.take(3 * db * F);
    q.w_o = a.take(db * db * T); q.b_o = a.take(db * F);
    q.ln2_g = a.take(db * F); q.ln2_b = a.take(db * F);
    q.w_ff1 = a.take(r * db * db * T); q.b_ff1 = a.take(r * db * F);
    q.w_ff2 = a.take(db * (r * db + dc) * T); q.b_ff2 = a.take(db * F); q.b_ff2_rj = a.take(db * F);
    if (b == 0) {
      p.blk0 = q;
      p.blk_stride = a.off - first;
    }
  }
  if (d->n_blocks == 0) p.blk_stride = 0;
  p.ln_f_g = a.take(db * F); p.ln_f_b = a.take(db * F);
  p.w_out = a.take(D * db * T); p.b_out = a.take(D * F); p.sigma_delta = a.take(D * F);
  p.tmp = a.take(db * db * T + E * F);
  p.total = a.off;
  return p;
}

struct Workspace {
  int64_t n, n_pad, ldst;
  uint64_t lo, hi, pos, gpos, flags, blocks, blocks_out, rope, krope, U, st, h, a, q, k, vt, o,
      f, total;
};

Workspace workspace_layout(const cr_dims* d, const cr_kv_layout* l, int64_t N) {
  const size_t T = esize(l->dtype);
  const int64_t S = 2LL * l->n_layers * l->n_kv_heads;
  const int64_t dc = d->d_c, db = d->d_b, r = d->ffn_mult, dhd = db / d->n_heads;
  const int64_t kc_pad = round_up(S * d->d_seg, 64);
  Workspace w;
  w.n = N;
  w.n_pad = round_up(std::max<int64_t>(N, 1), 128);
  w.ldst = dc;
  Arena a;
  w.lo = a.take(N * 4); w.hi = a.take(N * 4); w.pos = a.take(N * 4);
  w.gpos = a.take(N * 4); w.flags = a.take(N * 4);
  w.blocks = a.take(N * 4);                           // device copy of a paged block table
  w.blocks_out = a.take(N * 4);                       // ... and of the destination's
  w.rope = a.take(std::max<int64_t>(N, 1) * (dhd / 2) * 8);
  w.krope = a.take(N * (l->head_dim / 2) * 8);        // global key placement table
  w.U = a.take(N * kc_pad * T);
  w.st = a.take(N * w.ldst * T);
  w.h = a.take(N * db * T);
  w.a = a.take(N * db * T);
  w.q = a.take(N * db * T);
  w.k = a.take(w.n_pad * db * T);     // key rows padded like V^T
  w.vt = a.take(db * w.n_pad * T);
  w.o = a.take(N * db * T);
  w.f = a.take(N * r * db * T);
  w.total = a.off;
  return w;
}

// ------------------------------------------------------------- profiling
struct Profiler {
  std::mutex mu;
  std::vector<hipEvent_t> ev;        // 2 per launch slot
  std::vector<std::string> cls;      // class of each used slot
  std::vector<char> valid;           // the slot's events were recorded
  int used = 0;
  std::atomic<bool> on{false};       // read without the lock on every launch
};
Profiler& prof() {
  static Profiler p;
  return p;
}

// Launch `f` on stream s, bracketed by events when profiling is enabled.
// While a slot is in use the profiler's lock is held, so a concurrent
// cr_profile_enable cannot destroy its events; a stage that fails leaves its
// slot marked invalid (its events may never be recorded).
template <typename F>
hipError_t timed(const char* name, hipStream_t s, F&& f) {
  Profiler& P = prof();
  if (!P.on) return f();
  std::unique_lock<std::mutex> g(P.mu);
  if (!P.on || P.used >= (int)P.ev.size() / 2) {
    g.unlock();
    return f();
  }
  const int slot = P.used++;
  P.cls.emplace_back(name);
  P.valid.push_back(0);
  const hipEvent_t e0 = P.ev[2 * slot], e1 = P.ev[2 * slot + 1];
  LaunchEvents& le = launch_events();
  le.start = e0;
  le.stop = e1;
  hipError_t e = f();
  if (e == hipSuccess && le.start) {   // the stage launched nothing: an empty interval
    e = hipEventRecord(e0, s);
    if (e == hipSuccess) e = hipEventRecord(e1, s);
  }
  le = LaunchEvents{};
  P.valid[slot] = e == hipSuccess;
  return e;
}

#define CR_TRY(...)                                 \
  do {                                            \
    if ((__VA_ARGS__) != hipSuccess) return CR_ERR_LAUNCH; \
  } while (0)

template <typename T>
cr_status prepare_impl(const cr_dims* d, const cr_kv_layout* l, const char* blob, char* out,
                       hipStream_t s) {
  uint64_t total = 0;
  const std::vector<Tensor> c = canonical(d, l, &total);
  const Prepared p = prepared_layout(d, l);
  auto src = [&](const std::string& n) -> const T* {
    for (const Tensor& t : c)
      if (t.name == n) return reinterpret_cast<const T*>(blob + t.off);
    return nullptr;
  };
  auto srcf = [&](const std::string& n) -> const float* {
    for (const Tensor& t : c)
      if (t.name == n) return reinterpret_cast<const float*>(blob + t.off);
    return nullptr;
  };
  const int S = 2 * l->n_layers * l->n_kv_heads, dh = l->head_dim, D = S * dh;
  const int dc = d->d_c, db = d->d_b, E = d->d_model, r = d->ffn_mult, ds = d->d_seg;
  auto mat = [&](const std::string& n, uint64_t dst, int in, int outn, int in_pad) {
    return cr::transpose_convert<T, T>(src(n), reinterpret_cast<T*>(out + dst), 1, in, outn, outn,
                                       in_pad, nullptr, s);
  };
  auto vec = [&](const std::string& n, uint64_t dst, int len) {
    return cr::convert_f32<T>(src(n), reinterpret_cast<float*>(out + dst), len, len, 1, 0, 0, s);
  };
  // 1/sigma_stale folded into the per-segment projections
  CR_TRY(cr::transpose_convert<T, T>(src("w_seg"), reinterpret_cast<T*>(out + p.w_seg), S, dh, ds,
                                     32, dh, srcf("sigma_stale"), s));
  CR_TRY(cr::convert_f32<T>(src("b_seg"), reinterpret_cast<float*>(out + p.b_seg), ds, 32, S, ds,
                            32, s));
  CR_TRY(mat("w_cmp", p.w_cmp, (int)p.kc, dc, (int)p.kc_pad));
  CR_TRY(vec("b_cmp", p.b_cmp, dc));
  CR_TRY(vec("ln_enc_g", p.ln_enc_g, dc));
  CR_TRY(vec("ln_enc_b", p.ln_enc_b, dc));
  // token projection composed into the fusion (both affine, nothing between
  // them): the s columns of W_fuse^T first (the e columns zero-filled), then
  // (W_tok W_fuse_t)^T = W_fuse_t^T W_tok^T into the e columns, formed by the
  // library GEMM from W_fuse_t^T (in tmp) and W_tok (canonical [E][d_b]),
  // rounded once to the storage type; the bias is composed in fp32
  // (the reinjecting copy's s columns take W_fuse_s + W_inj_0, summed in
  // fp32 and rounded once, and its bias b_inj_0 too)
  T* wft = reinterpret_cast<T*>(out + p.tmp);
  float* zero = reinterpret_cast<float*>(out + p.tmp + (uint64_t)db * db * sizeof(T));
  const T* wfuse_t = src("w_fuse") + (int64_t)dc * db;
  CR_TRY(cr::transpose_convert<T, T>(wfuse_t, wft, 1, db, db, db, db, nullptr, s));
  CR_TRY(cr::convert_f32<T>(src("b_tok"), zero, 0, E, 1, 0, 0, s));
  for (int v = 0; v < 2; ++v) {
    const bool rjv = v == 1;
    if (rjv && d->n_blocks == 0) break;
    T* wf = reinterpret_cast<T*>(out + (rjv ? p.w_fuse_rj : p.w_fuse));
    CR_TRY(cr::transpose_into<T>(src("w_fuse"), rjv ? src("blk0.w_inj") : nullptr, wf, dc + E, dc,
                                 db, s));
    CR_TRY(cr::gemm_bias<T>(wft, db, src("w_tok"), db, db, E, db, wf + dc, dc + E, zero, nullptr,
                            0, false, s));
    CR_TRY(cr::compose_bias<T>(src("b_tok"), wfuse_t, db, src("b_fuse"),
                               rjv ? src("blk0.b_inj") : nullptr,
                               reinterpret_cast<float*>(out + (rjv ? p.b_fuse_rj : p.b_fuse)), db,
                               db, s));
  }
  for (int b = 0; b < d->n_blocks; ++b) {
    const std::string q = "blk" + std::to_string(b) + ".";
    const BlockP B = p.blk(b);
    CR_TRY(vec(q + "ln1_g", B.ln1_g, db));
    CR_TRY(vec(q + "ln1_b", B.ln1_b, db));
    CR_TRY(mat(q + "w_qkv", B.w_qkv, db, 3 * db, db));
    CR_TRY(vec(q + "b_qkv", B.b_qkv, 3 * db));
    CR_TRY(mat(q + "w_o", B.w_o, db, db, db));
    CR_TRY(vec(q + "b_o", B.b_o, db));
    CR_TRY(vec(q + "ln2_g", B.ln2_g, db));
    CR_TRY(vec(q + "ln2_b", B.ln2_b, db));
    CR_TRY(mat(q + "w_ff1", B.w_ff1, db, r * db, db));
    CR_TRY(vec(q + "b_ff1", B.b_ff1, r * db));
    // FFN2 rows [W_ff2 | W_inj_{b+1}] (zeros after the last block), biases
    // b_ff2 and b_ff2 + b_inj_{b+1}
    CR_TRY(mat(q + "w_ff2", B.w_ff2, r * db, db, r * db + dc));
    CR_TRY(vec(q + "b_ff2", B.b_ff2, db));
    const std::string nq = "blk" + std::to_string(b + 1) + ".";
    const bool has_next = b + 1 < d->n_blocks;
    if (has_next)
      CR_TRY(cr::transpose_into<T>(src(nq + "w_inj"), nullptr,
                                   reinterpret_cast<T*>(out + B.w_ff2) + (int64_t)r * db,
                                   r * db + dc, dc, db, s));
    CR_TRY(cr::compose_bias<T>(nullptr, nullptr, 0, src(q + "b_ff2"),
                               has_next ? src(nq + "b_inj") : nullptr,
                               reinterpret_cast<float*>(out + B.b_ff2_rj), 0, db, s));
  }
  CR_TRY(vec("ln_f_g", p.ln_f_g, db));
  CR_TRY(vec("ln_f_b", p.ln_f_b, db));
  CR_TRY(mat("w_out", p.w_out, db, D, db));
  CR_TRY(vec("b_out", p.b_out, D));
  CR_TRY(cr::convert_f32<float>(srcf("sigma_delta"), reinterpret_cast<float*>(out + p.sigma_delta),
                                D, D, 1, 0, 0, s));
  return CR_OK;
}

// Options of one call, validated.
struct CallOpts {
  int mask = CR_MASK_BLOCK_CAUSAL;
  bool reinject = true;
  int expand_mode = cr::EXPAND_RESIDUAL | cr::EXPAND_K | cr::EXPAND_V;
  bool keep_first = false;
  bool place_keys = false;
  cr::KeyRope kr{};
  const int32_t* pos_offset = nullptr;
  const cr_kv_pages* pages = nullptr;
  void* kv_out = nullptr;                 // out of place: destination cache
  const cr_kv_layout* layout_out = nullptr;
  const cr_kv_pages* pages_out = nullptr;
};

template <typename T>
cr_status repair_impl(T* kv, const cr_kv_layout* l, const int32_t* off, int32_t n_chunks,
                      const int32_t* req, int32_t n_req, const T* emb, const cr_dims* d,
                      const char* prep, char* ws, int64_t N, const CallOpts& opt,
                      hipStream_t s) {
  const Prepared P = prepared_layout(d, l);
  const Workspace W = workspace_layout(d, l, N);
  const int M = (int)N;
  const int dc = d->d_c, db = d->d_b, E = d->d_model, r = d->ffn_mult, nh = d->n_heads;
  const int dhd = db / nh;
  const int S = 2 * l->n_layers * l->n_kv_heads, D = S * l->head_dim;
  const int64_t ldst = W.ldst;
  auto PT = [&](uint64_t o) { return reinterpret_cast<const T*>(prep + o); };
  auto PF = [&](uint64_t o) { return reinterpret_cast<const float*>(prep + o); };
  auto WT = [&](uint64_t o) { return reinterpret_cast<T*>(ws + o); };
  int* lo = reinterpret_cast<int*>(ws + W.lo);
  int* hi = reinterpret_cast<int*>(ws + W.hi);
  int* pos = reinterpret_cast<int*>(ws + W.pos);
  int* gpos = opt.place_keys ? reinterpret_cast<int*>(ws + W.gpos) : nullptr;
  int* flags = opt.keep_first ? reinterpret_cast<int*>(ws + W.flags) : nullptr;
  float2* rope = reinterpret_cast<float2*>(ws + W.rope);
  float2* krope = reinterpret_cast<float2*>(ws + W.krope);
  T *U = WT(W.U), *st = WT(W.st), *h = WT(W.h), *a = WT(W.a), *q = WT(W.q),
    *k = WT(W.k), *vt = WT(W.vt), *o = WT(W.o), *f = WT(W.f);
  const int B = d->n_blocks;
  cr::KvStrides ks{l->stride_layer, l->stride_kv, l->stride_token, l->stride_head,
                   l->n_kv_heads, l->head_dim};
  const float eps = d->ln_eps;
  if (opt.pages) {
    int* blocks = reinterpret_cast<int*>(ws + W.blocks);
    const int nb = (int)((N + opt.pages->block_size - 1) / opt.pages->block_size);
    CR_TRY(timed("block_table", s, [&] {
        return cr::copy_table(opt.pages->block_table, nb, blocks, s); }));
    ks.blocks = blocks;
    ks.block_shift = log2_int(opt.pages->block_size);
    ks.block = opt.pages->stride_block;
  }
  T* kv_out = static_cast<T*>(opt.kv_out);
  cr::KvStrides ks_out{};
  if (kv_out) {
    const cr_kv_layout* lo_ = opt.layout_out;
    ks_out = cr::KvStrides{lo_->stride_layer, lo_->stride_kv, lo_->stride_token, lo_->stride_head,
                           lo_->n_kv_heads, lo_->head_dim};
    if (opt.pages_out) {
      int* blocks = reinterpret_cast<int*>(ws + W.blocks_out);
      const int nb = (int)((N + opt.pages_out->block_size - 1) / opt.pages_out->block_size);
      CR_TRY(timed("block_table", s, [&] {
          return cr::copy_table(opt.pages_out->block_table, nb, blocks, s); }));
      ks_out.blocks = blocks;
      ks_out.block_shift = log2_int(opt.pages_out->block_size);
      ks_out.block = opt.pages_out->stride_block;
    }
  }

  // the schedule also writes the repair network's RoPE table of the positions
  CR_TRY(timed("schedule", s, [&] {
      return cr::chunk_schedule(off, n_chunks, req, n_req, opt.mask, opt.pos_offset, lo, hi, pos,
                                gpos, flags, s, rope, dhd, (double)d->rope_theta); }));
  if (opt.place_keys)
    CR_TRY(timed("key_rope_table", s, [&] {
        return cr::key_rope_table(krope, gpos, M, opt.kr, s); }));
  // StaleEncoder: per-segment projections, compression, LN_enc -> s = st[:, :d_c]
  CR_TRY(timed("compress_segments", s, [&] {
      return cr::compress_segments<T>(kv, ks, l->n_layers, PT(P.w_seg), PF(P.b_seg), U, P.kc_pad,
                                  d->d_seg, M, s); }));
  CR_TRY(timed("gemm_compress", s, [&] {
      return cr::gemm_bias<T>(U, P.kc_pad, PT(P.w_cmp), P.kc_pad, M, dc, (int)P.kc_pad, st, ldst,
                          PF(P.b_cmp), nullptr, 0, false, s); }));
  CR_TRY(timed("layernorm", s, [&] {
      return cr::layernorm<T>(st, ldst, st, ldst, PF(P.ln_enc_g), PF(P.ln_enc_b), M, dc, eps, s); }));
  // reinjections P_b(s) (none for the entrance-only variant) ride on the
  // products before them: block 0's on the fusion, block b's on block b-1's
  // FFN2 (extra K columns of s)
  const bool rj = opt.reinject && B > 0;
  // token projection and fusion as one product of [s ; e] -> h^0 (+ P_0(s))
  CR_TRY(timed("gemm_fuse", s, [&] {
      return cr::gemm_bias_split<T>(st, ldst, dc, emb, E, PT(rj ? P.w_fuse_rj : P.w_fuse), dc + E,
                                    M, db, dc + E, h, db, PF(rj ? P.b_fuse_rj : P.b_fuse), nullptr,
                                    0, s); }));
  // h holds x_b = h^{b-1} + P_b(s) on entry to block b, h^B after the last block
  const int kff = r * db;   // FFN2 inner width; its prepared rows are kff + d_c long
  for (int b = 0; b < B; ++b) {
    const BlockP Bk = P.blk(b);
    const bool next_rj = rj && b + 1 < B;
    CR_TRY(timed("layernorm", s, [&] {
        return cr::layernorm<T>(h, db, a, db, PF(Bk.ln1_g), PF(Bk.ln1_b), M, db, eps, s); }));
    CR_TRY(timed("gemm_qkv", s, [&] {
        return cr::gemm_qkv<T>(a, db, PT(Bk.w_qkv), M, db, db, dhd, q, k, vt, W.n_pad, PF(Bk.b_qkv),
                           rope, s); }));
    CR_TRY(timed("attention", s, [&] {
        return cr::attention<T>(q, k, vt, o, M, db, nh, dhd, W.n_pad, lo, hi, s); }));
    CR_TRY(timed("gemm_oproj", s, [&] {
        return cr::gemm_bias<T>(o, db, PT(Bk.w_o), db, M, db, db, h, db, PF(Bk.b_o), h, db, false, s); }));
    CR_TRY(timed("layernorm", s, [&] {
        return cr::layernorm<T>(h, db, a, db, PF(Bk.ln2_g), PF(Bk.ln2_b), M, db, eps, s); }));
    CR_TRY(timed("gemm_ffn1", s, [&] {
        return cr::gemm_bias<T>(a, db, PT(Bk.w_ff1), db, M, r * db, db, f, (int64_t)r * db,
                            PF(Bk.b_ff1), nullptr, 0, true, s); }));
    CR_TRY(timed("gemm_ffn2", s, [&] {
        if (next_rj)   // h^{b+1} + P_{b+1}(s) = h + [f ; s] [W_ff2 ; W_inj] + b_ff2 + b_inj
          return cr::gemm_bias_split<T>(f, kff, kff, st, ldst, PT(Bk.w_ff2), kff + dc, M, db,
                                        kff + dc, h, db, PF(Bk.b_ff2_rj), h, db, s);
        return cr::gemm_bias<T>(f, kff, PT(Bk.w_ff2), kff + dc, M, db, kff, h, db, PF(Bk.b_ff2), h,
                                db, false, s); }));
  }
  CR_TRY(timed("layernorm", s, [&] {
      return cr::layernorm<T>(h, db, a, db, PF(P.ln_f_g), PF(P.ln_f_b), M, db, eps, s); }));
  CR_TRY(timed("gemm_expand", s, [&] {
      return cr::gemm_expand<T>(a, db, PT(P.w_out), M, D, db, kv, ks, PF(P.b_out),
                            PF(P.sigma_delta), opt.expand_mode, flags,
                            opt.place_keys ? krope : nullptr, kv_out, ks_out, s); }));
  return CR_OK;
}

}  // namespace

extern "C" {

int32_t cr_version(void) { return CR_ABI_VERSION; }

const char* cr_status_string(cr_status s) {
  switch (s) {
    case CR_OK: return "ok";
    case CR_ERR_NULL: return "a required pointer is NULL";
    case CR_ERR_DIMS: return "unsupported repairer or cache dimensions";
    case CR_ERR_OFFSETS: return "malformed chunk_offsets or request_chunks";
    case CR_ERR_LAYOUT: return "cache strides overlap, are misaligned or negative";
    case CR_ERR_WORKSPACE: return "buffer too small or misaligned";
    case CR_ERR_DTYPE: return "unknown storage dtype";
    case CR_ERR_DEVICE: return "current device is not gfx950";
    case CR_ERR_LAUNCH: return "kernel launch failed";
    case CR_ERR_CAPACITY: return "descriptor table too small";
    default: return "unknown status";
  }
}

cr_status cr_weights_layout(const cr_dims* dims, const cr_kv_layout* layout,
                            cr_tensor_desc* entries, int32_t max_entries, int32_t* n_entries,
                            uint64_t* total_bytes) {
  if (!dims || !layout || !n_entries || !total_bytes) return CR_ERR_NULL;
  const cr_status st = check_dims(dims, layout);
  if (st != CR_OK) return st;
  uint64_t total = 0;
  const std::vector<Tensor> v = canonical(dims, layout, &total);
  *n_entries = (int32_t)v.size();
  *total_bytes = total;
  if (!entries) return CR_OK;
  if (max_entries < (int32_t)v.size()) return CR_ERR_CAPACITY;
  for (size_t i = 0; i < v.size(); ++i) {
    cr_tensor_desc& e = entries[i];
    std::memset(&e, 0, sizeof(e));
    std::strncpy(e.name, v[i].name.c_str(), CR_MAX_NAME - 1);
    e.dtype = v[i].dtype;
    e.ndim = (int32_t)v[i].shape.size();
    for (int k = 0; k < e.ndim; ++k) e.shape[k] = v[i].shape[k];
    e.offset_bytes = v[i].off;
    e.nbytes = v[i].nbytes;
  }
  return CR_OK;
}

cr_status cr_prepared_bytes(const cr_dims* dims, const cr_kv_layout* layout, uint64_t* bytes) {
  if (!dims || !layout || !bytes) return CR_ERR_NULL;
  const cr_status st = check_dims(dims, layout);
  if (st != CR_OK) return st;
  *bytes = prepared_layout(dims, layout).total;
  return CR_OK;
}

cr_status cr_workspace_bytes(const cr_dims* dims, const cr_kv_layout* layout, int64_t n_tokens,
                             uint64_t* bytes) {
  if (!dims || !layout || !bytes) return CR_ERR_NULL;
  const cr_status st = check_dims(dims, layout);
  if (st != CR_OK) return st;
  if (n_tokens < 0 || n_tokens >= ((int64_t)1 << 31) - 256) return CR_ERR_DIMS;
  *bytes = workspace_layout(dims, layout, n_tokens).total;
  return CR_OK;
}

cr_status cr_workspace_view(const cr_dims* dims, const cr_kv_layout* layout, int64_t n_tokens,
                            const char* name, uint64_t* offset_bytes, int64_t* row_stride) {
  if (!dims || !layout || !name || !offset_bytes || !row_stride) return CR_ERR_NULL;
  const cr_status st = check_dims(dims, layout);
  if (st != CR_OK) return st;
  if (n_tokens < 0 || n_tokens >= ((int64_t)1 << 31) - 256) return CR_ERR_DIMS;
  const Workspace w = workspace_layout(dims, layout, n_tokens);
  if (!std::strcmp(name, "s")) { *offset_bytes = w.st; *row_stride = w.ldst; }
  else if (!std::strcmp(name, "h")) { *offset_bytes = w.h; *row_stride = dims->d_b; }
  else if (!std::strcmp(name, "lnf")) { *offset_bytes = w.a; *row_stride = dims->d_b; }
  else return CR_ERR_DIMS;
  return CR_OK;
}

cr_status cr_prepare_weights(const cr_dims* dims, const cr_kv_layout* layout, const void* blob,
                             uint64_t blob_bytes, void* prepared, uint64_t prepared_bytes,
                             void* stream) {
  if (!dims || !layout || !blob || !prepared) return CR_ERR_NULL;
  cr_status st = check_dims(dims, layout);
  if (st != CR_OK) return st;
  uint64_t need = 0;
  canonical(dims, layout, &need);
  if (blob_bytes < need || !aligned(blob, ALIGN)) return CR_ERR_WORKSPACE;
  if (prepared_bytes < prepared_layout(dims, layout).total || !aligned(prepared, ALIGN))
    return CR_ERR_WORKSPACE;
  st = check_device();
  if (st != CR_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (layout->dtype == CR_DTYPE_BF16)
    return prepare_impl<bf16>(dims, layout, static_cast<const char*>(blob),
                              static_cast<char*>(prepared), s);
  return prepare_impl<float>(dims, layout, static_cast<const char*>(blob),
                             static_cast<char*>(prepared), s);
}

cr_status cr_chunk_schedule(const int32_t* chunk_offsets, int32_t n_chunks,
                            const int32_t* request_chunks, int32_t n_requests, int32_t* rows,
                            void* stream) {
  if (!rows) return CR_ERR_NULL;
  cr_status st = check_offsets(chunk_offsets, n_chunks, request_chunks, n_requests);
  if (st != CR_OK) return st;
  const int64_t N = chunk_offsets[n_chunks];
  if (N == 0) return CR_OK;
  st = check_device();
  if (st != CR_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (cr::chunk_schedule(chunk_offsets, n_chunks, request_chunks, n_requests,
                         CR_MASK_BLOCK_CAUSAL, nullptr, rows, rows + N, rows + 2 * N, nullptr,
                         nullptr, s) != hipSuccess)
    return CR_ERR_LAUNCH;
  return CR_OK;
}

void cr_default_options(cr_options* opt) {
  if (!opt) return;
  std::memset(opt, 0, sizeof(*opt));
  opt->mask = CR_MASK_BLOCK_CAUSAL;
  opt->reinject = 1;
  opt->residual = 1;
  opt->apply = CR_APPLY_KV;
  opt->keep_first_chunk = 0;
  opt->global_rope = nullptr;
  opt->position_offset = nullptr;
  opt->pages = nullptr;
  opt->kv_out = nullptr;
  opt->layout_out = nullptr;
  opt->pages_out = nullptr;
}

}  // extern "C"

namespace {

// A validated repair call.
struct Call {
  CallOpts opt;
  int64_t N = 0;
};

bool same_shape(const cr_kv_layout* a, const cr_kv_layout* b) {
  return a->n_layers == b->n_layers && a->n_kv_heads == b->n_kv_heads &&
         a->head_dim == b->head_dim && a->dtype == b->dtype;
}

// Host-side validation of one cr_repair_ex call (nothing is enqueued).
// static_ws: the workspace is the library's static scratch (workspace is
// null here; workspace_bytes is the scratch size).
cr_status validate_call(const void* kv, const cr_kv_layout* layout, const int32_t* chunk_offsets,
                        int32_t n_chunks, const int32_t* request_chunks, int32_t n_requests,
                        const void* token_embeds, const cr_dims* dims, const void* prepared,
                        uint64_t prepared_bytes, const void* workspace, uint64_t workspace_bytes,
                        const cr_options& o, Call* c, bool static_ws = false) {
  if (!kv || !layout || !token_embeds || !dims || !prepared || (!workspace && !static_ws))
    return CR_ERR_NULL;
  cr_status st = check_dims(dims, layout);
  if (st != CR_OK) return st;
  st = check_offsets(chunk_offsets, n_chunks, request_chunks, n_requests);
  if (st != CR_OK) return st;
  CallOpts& opt = c->opt;
  if (o.mask < CR_MASK_BLOCK_CAUSAL || o.mask > CR_MASK_BLOCK_DIAGONAL) return CR_ERR_DIMS;
  if ((o.reinject != 0 && o.reinject != 1) || (o.residual != 0 && o.residual != 1) ||
      (o.keep_first_chunk != 0 && o.keep_first_chunk != 1))
    return CR_ERR_DIMS;
  if (o.apply < CR_APPLY_KV || o.apply > CR_APPLY_V) return CR_ERR_DIMS;
  opt.mask = o.mask;
  opt.reinject = o.reinject == 1;
  opt.expand_mode = (o.residual ? cr::EXPAND_RESIDUAL : 0) |
                    (o.apply != CR_APPLY_V ? cr::EXPAND_K : 0) |
                    (o.apply != CR_APPLY_K ? cr::EXPAND_V : 0);
  opt.keep_first = o.keep_first_chunk == 1;
  if (o.global_rope) {
    if (layout->head_dim > 128) return CR_ERR_DIMS;
    st = key_rope_of(o.global_rope, layout->head_dim, &opt.kr);
    if (st != CR_OK) return st;
    st = check_positions(chunk_offsets, n_chunks, request_chunks, n_requests, o.position_offset);
    if (st != CR_OK) return st;
    opt.place_keys = true;
    opt.pos_offset = o.position_offset;
  }
  const int64_t N = chunk_offsets[n_chunks];
  if (N >= ((int64_t)1 << 31) - 256) return CR_ERR_DIMS;
  if (o.pages) {
    st = check_pages(layout, o.pages, N);
    opt.pages = o.pages;
  } else {
    st = check_layout(layout, N);
  }
  if (st != CR_OK) return st;
  if (!aligned(kv, 16) || !aligned(token_embeds, 16)) return CR_ERR_LAYOUT;
  if (o.kv_out) {
    if (!o.layout_out) return CR_ERR_NULL;
    if (!same_shape(layout, o.layout_out)) return CR_ERR_LAYOUT;
    st = o.pages_out ? check_pages(o.layout_out, o.pages_out, N) : check_layout(o.layout_out, N);
    if (st != CR_OK) return st;
    if (!aligned(o.kv_out, 16) || o.kv_out == kv) return CR_ERR_LAYOUT;
    opt.kv_out = o.kv_out;
    opt.layout_out = o.layout_out;
    opt.pages_out = o.pages_out;
  }
  if (prepared_bytes < prepared_layout(dims, layout).total || !aligned(prepared, ALIGN))
    return CR_ERR_WORKSPACE;
  if (workspace_bytes < workspace_layout(dims, layout, N).total ||
      (!static_ws && !aligned(workspace, ALIGN)))
    return CR_ERR_WORKSPACE;
  c->N = N;
  return CR_OK;
}

cr_status enqueue_call(void* kv, const cr_kv_layout* layout, const int32_t* chunk_offsets,
                       int32_t n_chunks, const int32_t* request_chunks, int32_t n_requests,
                       const void* token_embeds, const cr_dims* dims, const void* prepared,
                       void* workspace, const Call& c, hipStream_t s) {
  if (c.N == 0) return CR_OK;
  if (layout->dtype == CR_DTYPE_BF16)
    return repair_impl<bf16>(static_cast<bf16*>(kv), layout, chunk_offsets, n_chunks,
                             request_chunks, n_requests, static_cast<const bf16*>(token_embeds),
                             dims, static_cast<const char*>(prepared),
                             static_cast<char*>(workspace), c.N, c.opt, s);
  return repair_impl<float>(static_cast<float*>(kv), layout, chunk_offsets, n_chunks,
                            request_chunks, n_requests, static_cast<const float*>(token_embeds),
                            dims, static_cast<const char*>(prepared),
                            static_cast<char*>(workspace), c.N, c.opt, s);
}

// staging of the pipeline: per slot the cache [L][2][n][H][d_h] and the
// embeddings [n][d_model] of max_tokens tokens
struct Staging {
  uint64_t kv_bytes, emb_bytes, slot_bytes;
};
Staging staging_layout(const cr_dims* d, const cr_kv_layout* l, int64_t max_tokens) {
  Staging g;
  const uint64_t T = esize(l->dtype);
  g.kv_bytes = align_up((uint64_t)2 * l->n_layers * max_tokens * l->n_kv_heads * l->head_dim * T);
  g.emb_bytes = align_up((uint64_t)max_tokens * d->d_model * T);
  g.slot_bytes = g.kv_bytes + g.emb_bytes;
  return g;
}

}  // namespace

// Workspace of cr_repair_static: a device array of the library.  Every GPU
// that loads the library holds its own copy until the process ends.  Host
// code never uses this name as an address (on the host it only stands for
// the symbol): each device's copy is found once through hipGetSymbolAddress
// with that device current, and that address is what the kernels receive.
static __device__ __align__(256) char scratch[CR_STATIC_SCRATCH_BYTES];

namespace {

// This GPU's address of the scratch array, looked up on the first call made
// with the device current and kept per device.
cr_status scratch_address(void** out) {
  static std::mutex mu;
  static void* addr[64] = {};
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return CR_ERR_DEVICE;
  std::lock_guard<std::mutex> g(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return CR_ERR_DEVICE;
    if (!aligned(p, ALIGN)) return CR_ERR_DEVICE;
    addr[dev] = p;
  }
  *out = addr[dev];
  return CR_OK;
}

}  // namespace

struct cr_pipeline_s {
  hipEvent_t copied[2] = {nullptr, nullptr};
  hipEvent_t done[2] = {nullptr, nullptr};
  bool used[2] = {false, false};  // done[b] recorded by this or an earlier call
};

extern "C" {

cr_status cr_repair_ex(void* kv, const cr_kv_layout* layout, const int32_t* chunk_offsets,
                       int32_t n_chunks, const int32_t* request_chunks, int32_t n_requests,
                       const void* token_embeds, const cr_dims* dims, const void* prepared,
                       uint64_t prepared_bytes, void* workspace, uint64_t workspace_bytes,
                       void* stream, const cr_options* options) {
  if (!options) return CR_ERR_NULL;
  Call c;
  cr_status st = validate_call(kv, layout, chunk_offsets, n_chunks, request_chunks, n_requests,
                               token_embeds, dims, prepared, prepared_bytes, workspace,
                               workspace_bytes, *options, &c);
  if (st != CR_OK) return st;
  if (c.N == 0) return CR_OK;
  st = check_device();
  if (st != CR_OK) return st;
  return enqueue_call(kv, layout, chunk_offsets, n_chunks, request_chunks, n_requests,
                      token_embeds, dims, prepared, workspace, c,
                      reinterpret_cast<hipStream_t>(stream));
}

cr_status cr_pipeline_create(cr_pipeline* pipeline) {
  if (!pipeline) return CR_ERR_NULL;
  cr_pipeline p = new (std::nothrow) cr_pipeline_s;
  if (!p) return CR_ERR_DEVICE;
  for (int i = 0; i < 2; ++i) {
    if (hipEventCreateWithFlags(&p->copied[i], hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&p->done[i], hipEventDisableTiming) != hipSuccess) {
      cr_pipeline_destroy(p);
      return CR_ERR_DEVICE;
    }
  }
  *pipeline = p;
  return CR_OK;
}

cr_status cr_pipeline_destroy(cr_pipeline p) {
  if (!p) return CR_ERR_NULL;
  // teardown: a failed destroy leaves nothing the caller could act on
  for (int i = 0; i < 2; ++i) {
    if (p->copied[i]) (void)hipEventDestroy(p->copied[i]);
    if (p->done[i]) (void)hipEventDestroy(p->done[i]);
  }
  delete p;
  return CR_OK;
}

cr_status cr_pipeline_staging_bytes(const cr_dims* dims, const cr_kv_layout* layout,
                                    int64_t max_tokens, uint64_t* bytes) {
  if (!dims || !layout || !bytes) return CR_ERR_NULL;
  const cr_status st = check_dims(dims, layout);
  if (st != CR_OK) return st;
  if (max_tokens < 0 || max_tokens >= ((int64_t)1 << 31) - 256) return CR_ERR_DIMS;
  *bytes = 2 * staging_layout(dims, layout, max_tokens).slot_bytes;
  return CR_OK;
}

cr_status cr_repair_pipelined(cr_pipeline pipeline, const cr_pipeline_item* items,
                              int32_t n_items, const cr_dims* dims, const cr_kv_layout* layout,
                              const void* prepared, uint64_t prepared_bytes, void* staging,
                              uint64_t staging_bytes, int64_t max_tokens, void* workspace,
                              uint64_t workspace_bytes, const cr_options* options,
                              void* copy_stream, void* compute_stream) {
  if (!pipeline || !dims || !layout || !staging || !workspace) return CR_ERR_NULL;
  if (n_items < 0) return CR_ERR_DIMS;
  if (n_items > 0 && !items) return CR_ERR_NULL;
  if (copy_stream == compute_stream) return CR_ERR_DIMS;
  cr_status st = check_dims(dims, layout);
  if (st != CR_OK) return st;
  if (max_tokens < 0 || max_tokens >= ((int64_t)1 << 31) - 256) return CR_ERR_DIMS;
  const Staging g = staging_layout(dims, layout, max_tokens);
  if (staging_bytes < 2 * g.slot_bytes || !aligned(staging, ALIGN)) return CR_ERR_WORKSPACE;
  cr_options base;
  cr_default_options(&base);
  if (options) base = *options;
  base.pages = nullptr;
  // validate every item against its own staging slot before enqueueing anything
  std::vector<Call> calls(n_items);
  std::vector<cr_kv_layout> lays(n_items);
  for (int i = 0; i < n_items; ++i) {
    const cr_pipeline_item& it = items[i];
    if (!it.kv_host || !it.embeds_host || !it.chunk_offsets || !it.kv_out || !it.layout_out)
      return CR_ERR_NULL;
    st = check_offsets(it.chunk_offsets, it.n_chunks, nullptr, 1);
    if (st != CR_OK) return st;
    const int64_t n = it.chunk_offsets[it.n_chunks];
    if (n > max_tokens) return CR_ERR_WORKSPACE;
    const int64_t sT = (int64_t)layout->n_kv_heads * layout->head_dim;
    lays[i] = cr_kv_layout{layout->n_layers, layout->n_kv_heads, layout->head_dim,
                           layout->dtype, 2 * n * sT, n * sT, sT, layout->head_dim};
    cr_options o = base;
    o.kv_out = it.kv_out;
    o.layout_out = it.layout_out;
    o.pages_out = it.pages_out;
    o.position_offset = &it.position_offset;
    char* slot = static_cast<char*>(staging) + (i & 1) * g.slot_bytes;
    st = validate_call(slot, &lays[i], it.chunk_offsets, it.n_chunks, nullptr, 1,
                       slot + g.kv_bytes, dims, prepared, prepared_bytes, workspace,
                       workspace_bytes, o, &calls[i]);
    if (st != CR_OK) return st;
  }
  if (n_items == 0) return CR_OK;
  st = check_device();
  if (st != CR_OK) return st;
  hipStream_t cs = reinterpret_cast<hipStream_t>(copy_stream);
  hipStream_t ks = reinterpret_cast<hipStream_t>(compute_stream);
  const uint64_t T = esize(layout->dtype);
  for (int i = 0; i < n_items; ++i) {
    const cr_pipeline_item& it = items[i];
    const int b = i & 1;
    char* slot = static_cast<char*>(staging) + b * g.slot_bytes;
    const int64_t n = calls[i].N;
    // the slot is refilled only after the repair that read it has finished
    // (in this call or in an earlier one on the same handle)
    if (pipeline->used[b] && hipStreamWaitEvent(cs, pipeline->done[b], 0) != hipSuccess)
      return CR_ERR_LAUNCH;
    const uint64_t kvb = (uint64_t)2 * layout->n_layers * n * layout->n_kv_heads * layout->head_dim * T;
    const uint64_t eb = (uint64_t)n * dims->d_model * T;
    if (n > 0) {
      if (hipMemcpyAsync(slot, it.kv_host, kvb, hipMemcpyHostToDevice, cs) != hipSuccess ||
          hipMemcpyAsync(slot + g.kv_bytes, it.embeds_host, eb, hipMemcpyHostToDevice, cs) !=
              hipSuccess)
        return CR_ERR_LAUNCH;
    }
    if (hipEventRecord(pipeline->copied[b], cs) != hipSuccess ||
        hipStreamWaitEvent(ks, pipeline->copied[b], 0) != hipSuccess)
      return CR_ERR_LAUNCH;
    st = enqueue_call(slot, &lays[i], it.chunk_offsets, it.n_chunks, nullptr, 1,
                      slot + g.kv_bytes, dims, prepared, workspace, calls[i], ks);
    if (st != CR_OK) return st;
    if (hipEventRecord(pipeline->done[b], ks) != hipSuccess) return CR_ERR_LAUNCH;
    pipeline->used[b] = true;
  }
  return CR_OK;
}

cr_status cr_repair(void* kv, const cr_kv_layout* layout, const int32_t* chunk_offsets,
                    int32_t n_chunks, const int32_t* request_chunks, int32_t n_requests,
                    const void* token_embeds, const cr_dims* dims, const void* prepared,
                    uint64_t prepared_bytes, void* workspace, uint64_t workspace_bytes,
                    void* stream) {
  cr_options o;
  cr_default_options(&o);
  return cr_repair_ex(kv, layout, chunk_offsets, n_chunks, request_chunks, n_requests,
                      token_embeds, dims, prepared, prepared_bytes, workspace, workspace_bytes,
                      stream, &o);
}

cr_status cr_repair_static(void* kv, const cr_kv_layout* layout, const int32_t* chunk_offsets,
                           int32_t n_chunks, const int32_t* request_chunks, int32_t n_requests,
                           const void* token_embeds, const cr_dims* dims, const void* prepared,
                           uint64_t prepared_bytes, void* stream) {
  cr_options o;
  cr_default_options(&o);
  Call c;
  cr_status st = validate_call(kv, layout, chunk_offsets, n_chunks, request_chunks, n_requests,
                               token_embeds, dims, prepared, prepared_bytes, nullptr,
                               CR_STATIC_SCRATCH_BYTES, o, &c, /*static_ws=*/true);
  if (st != CR_OK) return st;
  if (c.N == 0) return CR_OK;
  st = check_device();
  if (st != CR_OK) return st;
  void* ws = nullptr;
  st = scratch_address(&ws);
  if (st != CR_OK) return st;
  return enqueue_call(kv, layout, chunk_offsets, n_chunks, request_chunks, n_requests,
                      token_embeds, dims, prepared, ws, c, reinterpret_cast<hipStream_t>(stream));
}

// workspace of cr_rotate_keys: lo, hi, pos, gpos, block table (int32 each)
// and the (cos, sin) table
static uint64_t rotate_ws_bytes(const cr_kv_layout* l, int64_t N) {
  return align_up(5 * (uint64_t)N * 4) + align_up((uint64_t)N * (l->head_dim / 2) * 8);
}

cr_status cr_rotate_workspace_bytes(const cr_kv_layout* layout, int64_t n_tokens,
                                    uint64_t* bytes) {
  if (!layout || !bytes) return CR_ERR_NULL;
  if (n_tokens < 0 || n_tokens >= ((int64_t)1 << 31) - 256) return CR_ERR_DIMS;
  if (layout->head_dim < 32 || layout->head_dim > 256 || layout->head_dim % 32) return CR_ERR_DIMS;
  *bytes = rotate_ws_bytes(layout, n_tokens);
  return CR_OK;
}

cr_status cr_rotate_keys(void* kv, const cr_kv_layout* layout, const int32_t* chunk_offsets,
                         int32_t n_chunks, const int32_t* request_chunks, int32_t n_requests,
                         const cr_rope* rope, const int32_t* position_offset, int32_t inverse,
                         const cr_kv_pages* pages, void* workspace, uint64_t workspace_bytes,
                         void* stream) {
  if (!kv || !layout || !rope || !workspace) return CR_ERR_NULL;
  if (layout->n_layers < 1 || layout->n_kv_heads < 1 || layout->head_dim < 32 ||
      layout->head_dim > 256 || layout->head_dim % 32)
    return CR_ERR_DIMS;
  if (layout->dtype != CR_DTYPE_BF16 && layout->dtype != CR_DTYPE_F32) return CR_ERR_DTYPE;
  if (inverse != 0 && inverse != 1) return CR_ERR_DIMS;
  cr_status st = check_offsets(chunk_offsets, n_chunks, request_chunks, n_requests);
  if (st != CR_OK) return st;
  cr::KeyRope kr{};
  st = key_rope_of(rope, layout->head_dim, &kr);
  if (st != CR_OK) return st;
  st = check_positions(chunk_offsets, n_chunks, request_chunks, n_requests, position_offset);
  if (st != CR_OK) return st;
  const int64_t N = chunk_offsets[n_chunks];
  if (N >= ((int64_t)1 << 31) - 256) return CR_ERR_DIMS;
  st = pages ? check_pages(layout, pages, N) : check_layout(layout, N);
  if (st != CR_OK) return st;
  if (!aligned(kv, 16)) return CR_ERR_LAYOUT;
  if (workspace_bytes < rotate_ws_bytes(layout, N) || !aligned(workspace, ALIGN))
    return CR_ERR_WORKSPACE;
  if (N == 0) return CR_OK;
  st = check_device();
  if (st != CR_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  int* rows = static_cast<int*>(workspace);
  float2* tab = reinterpret_cast<float2*>(static_cast<char*>(workspace) + align_up(5 * (uint64_t)N * 4));
  cr::KvStrides ks{layout->stride_layer, layout->stride_kv, layout->stride_token,
                   layout->stride_head, layout->n_kv_heads, layout->head_dim};
  if (pages) {
    int* blocks = rows + 4 * N;
    if (cr::copy_table(pages->block_table, (int)((N + pages->block_size - 1) / pages->block_size),
                       blocks, s) != hipSuccess)
      return CR_ERR_LAUNCH;
    ks.blocks = blocks;
    ks.block_shift = log2_int(pages->block_size);
    ks.block = pages->stride_block;
  }
  if (cr::chunk_schedule(chunk_offsets, n_chunks, request_chunks, n_requests,
                         CR_MASK_BLOCK_CAUSAL, position_offset, rows, rows + N, rows + 2 * N,
                         rows + 3 * N, nullptr, s) != hipSuccess)
    return CR_ERR_LAUNCH;
  if (cr::key_rope_table(tab, rows + 3 * N, (int)N, kr, s) != hipSuccess) return CR_ERR_LAUNCH;
  hipError_t e;
  if (layout->dtype == CR_DTYPE_BF16)
    e = cr::rotate_keys<bf16>(static_cast<bf16*>(kv), ks, layout->n_layers, (int)N, tab,
                              inverse == 1, rope->scale, s);
  else
    e = cr::rotate_keys<float>(static_cast<float*>(kv), ks, layout->n_layers, (int)N, tab,
                               inverse == 1, rope->scale, s);
  return e == hipSuccess ? CR_OK : CR_ERR_LAUNCH;
}

cr_status cr_profile_enable(int32_t max_launches) {
  if (max_launches < 0) return CR_ERR_DIMS;
  Profiler& P = prof();
  std::lock_guard<std::mutex> g(P.mu);
  for (hipEvent_t e : P.ev) (void)hipEventDestroy(e);   // teardown of the previous slots
  P.ev.clear();
  P.cls.clear();
  P.valid.clear();
  P.used = 0;
  P.on = false;
  if (max_launches == 0) return CR_OK;
  P.ev.resize(2 * (size_t)max_launches, nullptr);
  for (hipEvent_t& e : P.ev) {
    if (hipEventCreate(&e) != hipSuccess) {
      for (hipEvent_t& x : P.ev)
        if (x) (void)hipEventDestroy(x);   // teardown of a partial set
      P.ev.clear();
      return CR_ERR_DEVICE;
    }
  }
  P.on = true;
  return CR_OK;
}

cr_status cr_profile_read(cr_kernel_stat* stats, int32_t max_stats, int32_t* n_stats) {
  if (!n_stats) return CR_ERR_NULL;
  Profiler& P = prof();
  std::lock_guard<std::mutex> g(P.mu);
  std::vector<std::string> names;
  std::vector<int> launches;
  std::vector<double> total;
  cr_status st = CR_OK;
  for (int i = 0; i < P.used && st == CR_OK; ++i) {
    if (!P.valid[i]) continue;        // its stage failed: nothing was timed
    float ms = 0.f;
    if (hipEventSynchronize(P.ev[2 * i + 1]) != hipSuccess ||
        hipEventElapsedTime(&ms, P.ev[2 * i], P.ev[2 * i + 1]) != hipSuccess) {
      st = CR_ERR_LAUNCH;
      break;
    }
    size_t k = std::find(names.begin(), names.end(), P.cls[i]) - names.begin();
    if (k == names.size()) { names.push_back(P.cls[i]); launches.push_back(0); total.push_back(0); }
    launches[k] += 1;
    total[k] += ms;
  }
  // the slots are free again whatever happened
  P.used = 0;
  P.cls.clear();
  P.valid.clear();
  if (st != CR_OK) return st;
  *n_stats = (int32_t)names.size();
  if (!stats) return CR_OK;
  if (max_stats < (int32_t)names.size()) return CR_ERR_CAPACITY;
  for (size_t k = 0; k < names.size(); ++k) {
    std::memset(&stats[k], 0, sizeof(cr_kernel_stat));
    std::strncpy(stats[k].name, names[k].c_str(), sizeof(stats[k].name) - 1);
    stats[k].launches = launches[k];
    stats[k].total_ms = total[k];
  }
  return CR_OK;
}

}  // extern "C"
