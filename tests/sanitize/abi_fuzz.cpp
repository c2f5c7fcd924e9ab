// Host-side fuzz of the CacheRepair C ABI's argument validation, built with
// AddressSanitizer and UndefinedBehaviorSanitizer on the host pass and
// linked against launchers that always fail (no kernel exists in this
// build).  Every call here is made with fake, never dereferenced device
// addresses: valid calls end at the device check (no GPU), invalid ones at
// their validation error.  The sanitizers report any out-of-bounds read of
// a host array (offsets, request chunks, block tables, frequency tables) or
// any undefined arithmetic in the layout checks.  Refuses to run where a GPU
// is visible.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

#include "cacherepair.h"

static std::mt19937_64 rng(20260402);
// The first value is the common, valid choice (taken 7 times in 8); the
// others, often invalid, share the rest.
static int64_t pick(std::initializer_list<int64_t> v) {
  if (rng() % 8 != 0) return *v.begin();
  return *(v.begin() + rng() % v.size());
}
static int64_t uni(int64_t a, int64_t b) { return a + (int64_t)(rng() % (uint64_t)(b - a + 1)); }

static int counts[16];
static void tally(cr_status s) { counts[-s < 16 && s <= 0 ? -s : 15]++; }

// Heap copies of exactly the elements a call may read, so a read past them
// is an AddressSanitizer report.
template <typename T>
struct Exact {
  T* p = nullptr;
  explicit Exact(const std::vector<T>& v) {
    if (!v.empty()) {
      p = new T[v.size()];
      std::memcpy(p, v.data(), v.size() * sizeof(T));
    }
  }
  ~Exact() { delete[] p; }
};

int main(int argc, char** argv) {
  int n_dev = 0;
  if (hipGetDeviceCount(&n_dev) == hipSuccess && n_dev > 0) {
    std::printf("abi_fuzz: a GPU is visible; this host-only check does not run there\n");
    return 0;
  }
  if (argc > 1 && std::strcmp(argv[1], "selftest") == 0) {
    // a read one element past a heap array: the instrumented build must stop here
    Exact<int32_t> a(std::vector<int32_t>(4, 1));
    volatile int32_t sink = a.p[4];
    std::printf("abi_fuzz: selftest read %d past the array without a report\n", (int)sink);
    return 0;
  }
  const long iters = argc > 1 ? std::atol(argv[1]) : 20000;
  void* const kv = reinterpret_cast<void*>(uintptr_t(1) << 40);      // never dereferenced
  void* const emb = reinterpret_cast<void*>(uintptr_t(2) << 40);
  void* const prep = reinterpret_cast<void*>(uintptr_t(3) << 40);
  void* const ws = reinterpret_cast<void*>(uintptr_t(4) << 40);
  void* const out = reinterpret_cast<void*>(uintptr_t(5) << 40);
  for (long it = 0; it < iters; ++it) {
    cr_dims d;
    d.d_model = (int32_t)pick({64, 128, 2048, 0, -64, 96, 1 << 30});
    d.d_seg = (int32_t)pick({8, 24, 32, 0, 33, -1});
    d.d_c = (int32_t)pick({64, 1024, 2048, 0, 4096, 100});
    d.d_b = (int32_t)pick({128, 1024, 2048, 0, 4096, 192});
    d.n_blocks = (int32_t)pick({0, 1, 8, 256, 257, -1});
    d.n_heads = (int32_t)pick({2, 1, 16, 32, 0, 3, -4});
    d.ffn_mult = (int32_t)pick({1, 4, 16, 0, 17});
    d.rope_theta = (float)pick({10000, 0, -1});
    d.ln_eps = rng() % 8 ? 1e-5f : -1.f;
    cr_kv_layout l;
    l.n_layers = (int32_t)pick({1, 2, 36, 0, -1, 1 << 20});
    l.n_kv_heads = (int32_t)pick({1, 2, 8, 0, -2});
    l.head_dim = (int32_t)pick({32, 64, 128, 256, 96, 16, 512, 0});
    l.dtype = (int32_t)pick({CR_DTYPE_BF16, CR_DTYPE_F32, 7, -1});
    const int64_t N = pick({0, 1, 5, 64, 4096, (int64_t)1 << 31, -3});
    const int64_t row = (int64_t)l.n_kv_heads * l.head_dim;
    l.stride_head = pick({l.head_dim, l.head_dim + 16, 0, -8, 12, (int64_t)1 << 61});
    l.stride_token = pick({row, row + 64, 2 * l.n_layers * row, 8, -16, (int64_t)1 << 62});
    l.stride_kv = pick({N * row, N * row + 8, 8, 0, INT64_MAX - 7});
    l.stride_layer = pick({2 * N * row, 2 * N * row + 24, 16, INT64_MIN + 8, (int64_t)1 << 55});
    // chunk offsets: well formed, decreasing, not starting at 0, or short
    const int32_t n_chunks = (int32_t)pick({1, 2, 7, 0, -1});
    std::vector<int32_t> off(n_chunks > 0 ? n_chunks + 1 : 1, 0);
    for (size_t i = 1; i < off.size(); ++i) off[i] = off[i - 1] + (int32_t)uni(0, 700);
    if (rng() % 8 == 0 && off.size() > 2) off[1] = off[2] + 1;
    if (rng() % 16 == 0) off[0] = 3;
    const int32_t n_req = (int32_t)pick({1, 2, 3, 0, -1});
    std::vector<int32_t> req(n_req > 0 ? n_req + 1 : 1, 0);
    for (size_t i = 1; i < req.size(); ++i) req[i] = std::min<int32_t>(req[i - 1] + (int32_t)uni(0, 3), n_chunks);
    if (!req.empty() && n_chunks > 0) req.back() = rng() % 8 ? n_chunks : n_chunks + 1;
    Exact<int32_t> offs(off), reqs(req);
    const int32_t* reqp = rng() % 3 ? reqs.p : nullptr;

    uint64_t bytes = 0;
    int32_t n_ent = 0;
    tally(cr_weights_layout(&d, &l, nullptr, 0, &n_ent, &bytes));
    tally(cr_prepared_bytes(&d, &l, &bytes));
    tally(cr_workspace_bytes(&d, &l, N, &bytes));
    int64_t stride = 0;
    tally(cr_workspace_view(&d, &l, N, rng() % 2 ? "s" : "x", &bytes, &stride));
    tally(cr_pipeline_staging_bytes(&d, &l, N, &bytes));
    tally(cr_rotate_workspace_bytes(&l, N, &bytes));
    const uint64_t big = pick({0, 1 << 20, (int64_t)1 << 40});
    tally(cr_repair(kv, &l, offs.p, n_chunks, reqp, n_req, emb, &d, prep, big, ws, big, nullptr));
    tally(cr_repair_static(kv, &l, offs.p, n_chunks, reqp, n_req, emb, &d, prep, big, nullptr));

    cr_options o;
    cr_default_options(&o);
    o.mask = (int32_t)pick({0, 1, 2, 3, 4, -1});
    o.apply = (int32_t)pick({0, 1, 2, 3});
    o.keep_first_chunk = (int32_t)pick({0, 1, 2});
    cr_rope rope{(double)pick({10000, 1000000, 0}), nullptr, rng() % 4 ? 1.0f : -1.0f};
    std::vector<float> freq((size_t)(l.head_dim > 0 && l.head_dim <= 512 ? l.head_dim / 2 : 1), 0.01f);
    Exact<float> freqs(freq);
    if (rng() % 2) rope.inv_freq = freqs.p;
    std::vector<int32_t> posoff(n_req > 0 ? n_req : 1, (int32_t)pick({0, 7, -1, INT32_MAX - 5}));
    Exact<int32_t> posoffs(posoff);
    if (rng() % 2) { o.global_rope = &rope; o.position_offset = posoffs.p; }
    const int32_t bsz = (int32_t)pick({16, 1, 1024, 3, 2048, 0});
    const int64_t total = off.back();
    const int64_t nb = bsz > 0 ? (total + bsz - 1) / bsz : 1;
    std::vector<int32_t> table((size_t)std::max<int64_t>(nb, 1));
    for (size_t i = 0; i < table.size(); ++i) table[i] = (int32_t)i;
    if (rng() % 8 == 0 && table.size() > 1) table[1] = table[0];         // duplicate block
    if (rng() % 8 == 0) table[0] = -1;
    Exact<int32_t> tables(table);
    cr_kv_pages pg{bsz, (int32_t)pick({(int64_t)table.size(), (int64_t)table.size() + 3, 1}),
                   pick({bsz * row, 8, -8}), tables.p};
    if (rng() % 3 == 0) o.pages = &pg;
    if (rng() % 4 == 0) { o.kv_out = out; o.layout_out = &l; }
    tally(cr_repair_ex(kv, &l, offs.p, n_chunks, reqp, n_req, emb, &d, prep, big, ws, big,
                       nullptr, &o));
    tally(cr_rotate_keys(kv, &l, offs.p, n_chunks, reqp, n_req, &rope, posoffs.p,
                         (int32_t)pick({0, 1, 2}), rng() % 2 ? &pg : nullptr, ws, big, nullptr));
    tally(cr_chunk_schedule(offs.p, n_chunks, reqp, n_req, static_cast<int32_t*>(ws), nullptr));
  }
  std::printf("abi_fuzz: %ld iterations; status counts:", iters);
  for (int i = 0; i < 16; ++i) std::printf(" %d:%d", -i, counts[i]);
  std::printf("\n");
  return 0;
}
