// Host-side checks of the library under AddressSanitizer, on the CPU.
//
// The library's sources are compiled for the host only and linked with a
// stand-in HIP runtime (fake_hip_runtime.cpp): "device" buffers are host
// allocations of exactly the size the library asks for, table uploads are
// memcpy, and kernel launches run nothing but have their launch shapes
// checked.  So every byte the host code writes -- pack plans and index maps,
// collector queues, workspace carving and the descriptor tables copied into
// the caller's workspace, the allocation-free call's scratch -- is checked by
// ASan against the buffer it belongs to, through every entry point and its
// error paths.  Test infrastructure only.  Prints "host checks ok" at the end.
#include <cstdint>
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "joynexus.h"

extern "C" long long jn_fake_launches;
extern "C" long long jn_fake_graph_launches;

namespace {

int g_checks = 0;

#define CHECK(cond)                                                          \
  do {                                                                       \
    ++g_checks;                                                              \
    if (!(cond)) {                                                           \
      std::fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      std::exit(2);                                                          \
    }                                                                        \
  } while (0)

struct Rng {
  uint64_t s;
  explicit Rng(uint64_t seed) : s(seed * 6364136223846793005ull + 1442695040888963407ull) {}
  uint32_t next() {
    s = s * 6364136223846793005ull + 1442695040888963407ull;
    return (uint32_t)(s >> 33);
  }
  int range(int lo, int hi) { return lo + (int)(next() % (uint32_t)(hi - lo + 1)); }
};

// Every "device" allocation: exactly n bytes, 256-byte aligned; released at exit.
std::vector<void*> g_allocs;
void* dev(size_t n) {
  void* p = nullptr;
  if (posix_memalign(&p, 256, n ? n : 1) != 0) std::abort();
  std::memset(p, 0, n ? n : 1);
  g_allocs.push_back(p);
  return p;
}

struct Group {
  std::vector<jn_request> req;
  std::vector<std::vector<int32_t>> lens;
  std::vector<jn_tenant> ten;
  jn_pack_opts opts{};
};

Group make_group(Rng& r, int G, int d, int max_reqs_per_tenant, int max_n, int max_len, int align) {
  Group g;
  g.opts.d_model = d;
  g.opts.align = align;
  g.ten.assign(G, jn_tenant{0x1234, d, 0});
  std::vector<int> order;
  for (int t = 0; t < G; ++t) {
    int k = r.range(1, max_reqs_per_tenant);
    for (int i = 0; i < k; ++i) order.push_back(t);
  }
  for (size_t i = order.size(); i > 1; --i) std::swap(order[i - 1], order[r.next() % i]);
  g.lens.resize(order.size());
  for (size_t i = 0; i < order.size(); ++i) {
    jn_request q{};
    q.tenant = order[i];
    q.n_samples = r.range(1, max_n);
    q.max_len = r.range(1, max_len);
    for (int s = 0; s < q.n_samples; ++s) g.lens[i].push_back(r.range(1, q.max_len));
    q.embeds = dev((size_t)q.n_samples * q.max_len * d * 2);
    g.req.push_back(q);
  }
  for (size_t i = 0; i < g.req.size(); ++i) g.req[i].lengths = g.lens[i].data();
  return g;
}

// G tenants, one request each of n samples of exactly len rows.
Group long_group(int d, int G, int n, int len) {
  Group g;
  g.opts.d_model = d;
  g.opts.align = 1;
  g.ten.assign(G, jn_tenant{0x1234, d, 0});
  g.lens.resize(G);
  for (int t = 0; t < G; ++t) {
    jn_request q{};
    q.tenant = t;
    q.n_samples = n;
    q.max_len = len;
    g.lens[t].assign(n, len);
    q.embeds = dev((size_t)n * len * d * 2);
    g.req.push_back(q);
  }
  for (int t = 0; t < G; ++t) g.req[t].lengths = g.lens[t].data();
  return g;
}

// One tenant, one request of n samples of exactly len rows.
Group fixed_group(int d, int n, int len) {
  Group g;
  g.opts.d_model = d;
  g.opts.align = 1;
  g.ten.assign(1, jn_tenant{0x1234, d, 0});
  g.lens.assign(1, std::vector<int32_t>(n, len));
  jn_request q{};
  q.tenant = 0;
  q.n_samples = n;
  q.max_len = len;
  q.embeds = dev((size_t)n * len * d * 2);
  q.lengths = g.lens[0].data();
  g.req.push_back(q);
  return g;
}

struct Packed {
  jn_pack_sizes sz{};
  jn_packed p{};
  void* maps = nullptr;
  void* tokens = nullptr;
};

Packed pack(jn_ctx* c, Group& g) {
  Packed k;
  CHECK(jn_pack_plan(g.req.data(), (int)g.req.size(), g.ten.data(), (int)g.ten.size(), &g.opts, &k.sz) == JN_OK);
  k.maps = dev(k.sz.map_bytes);
  k.tokens = dev(k.sz.token_bytes);
  // repeated uploads: the staging ring grows while copies are reported in
  // flight, then reuses its slots
  for (int rep = 0; rep < 100; ++rep)
    CHECK(jn_pack_group(c, g.req.data(), (int)g.req.size(), g.ten.data(), (int)g.ten.size(), &g.opts, k.maps,
                        k.sz.map_bytes, k.tokens, k.sz.token_bytes, &k.p) == JN_OK);
  // undersized buffers are refused
  jn_packed tmp{};
  CHECK(jn_pack_group(c, g.req.data(), (int)g.req.size(), g.ten.data(), (int)g.ten.size(), &g.opts, k.maps,
                      k.sz.map_bytes - 1, k.tokens, k.sz.token_bytes, &tmp) == JN_ENOSPACE);
  CHECK(jn_pack_group(c, g.req.data(), (int)g.req.size(), g.ten.data(), (int)g.ten.size(), &g.opts, k.maps,
                      k.sz.map_bytes, k.tokens, k.sz.token_bytes - 2, &tmp) == JN_ENOSPACE);
  return k;
}

// ------------------------------------------------------------- plans ---

void check_plans() {
  Rng r(1);
  for (int it = 0; it < 300; ++it) {
    const int aligns[] = {1, 2, 8, 16, 64, 128};
    Group g = make_group(r, r.range(1, 6), 64, 3, 9, 300, aligns[r.next() % 6]);
    jn_pack_sizes sz{};
    CHECK(jn_pack_plan(g.req.data(), (int)g.req.size(), g.ten.data(), (int)g.ten.size(), &g.opts, &sz) == JN_OK);
    std::vector<char> host(sz.map_bytes);
    jn_packed p{};
    CHECK(jn_pack_maps_host(g.req.data(), (int)g.req.size(), g.ten.data(), (int)g.ten.size(), &g.opts, host.data(),
                            host.size(), &p) == JN_OK);
    CHECK(p.cu_seqlens[0] == 0 && p.cu_seqlens[p.N] == p.T);
    std::vector<int> seen(p.N, 0);
    for (int k = 0; k < p.N; ++k) seen[p.tenant_perm[k]]++;
    for (int k = 0; k < p.N; ++k) CHECK(seen[k] == 1);
    CHECK(jn_pack_maps_host(g.req.data(), (int)g.req.size(), g.ten.data(), (int)g.ten.size(), &g.opts, host.data(),
                            host.size() - 1, &p) != JN_OK);
  }
  // error statuses
  Group g = make_group(r, 2, 64, 1, 3, 10, 1);
  jn_pack_sizes sz{};
  const int R = (int)g.req.size();
  CHECK(jn_pack_plan(nullptr, R, g.ten.data(), 2, &g.opts, &sz) == JN_EINVAL);
  CHECK(jn_pack_plan(g.req.data(), 0, g.ten.data(), 2, &g.opts, &sz) == JN_EINVAL);
  jn_pack_opts bad = g.opts;
  bad.align = 0;
  CHECK(jn_pack_plan(g.req.data(), R, g.ten.data(), 2, &bad, &sz) == JN_EINVAL);
  g.ten[1].prefix_sig = 99;
  CHECK(jn_pack_plan(g.req.data(), R, g.ten.data(), 2, &g.opts, &sz) == JN_EINCOMPAT);
  g.ten[1].prefix_sig = g.ten[0].prefix_sig;
  g.lens[0][0] = g.req[0].max_len + 1;
  CHECK(jn_pack_plan(g.req.data(), R, g.ten.data(), 2, &g.opts, &sz) == JN_ESHAPE);
  g.lens[0][0] = 1;
  g.req[0].tenant = 7;
  CHECK(jn_pack_plan(g.req.data(), R, g.ten.data(), 2, &g.opts, &sz) == JN_ESHAPE);
}

// --------------------------------------------------------- collector ---

void check_collector() {
  Rng r(2);
  for (int it = 0; it < 300; ++it) {
    jn_collector* c = nullptr;
    CHECK(jn_collector_create(&c, r.range(1, 40), r.range(0, 500)) == JN_OK);
    int64_t now = 0, id = 0, out = 0;
    const int n = r.range(0, 60);
    for (int i = 0; i < n; ++i) {
      now += r.range(0, 100);
      CHECK(jn_collector_submit(c, id++, (uint64_t)r.range(0, 2), 64, r.range(1, 12), now) == JN_OK);
      if (r.range(0, 2) == 0) {
        const int cap = r.range(1, 6);
        std::vector<int64_t> ids(cap);
        int32_t got = 0;
        jn_status st = jn_collector_poll(c, now + r.range(0, 600), ids.data(), cap, &got);
        CHECK(st == JN_OK || st == JN_ENOSPACE);
        if (st == JN_OK) out += got;
      }
    }
    // an arrival before the last queued request's is refused
    CHECK(jn_collector_submit(c, id++, 1, 64, 1, now) == JN_OK);
    CHECK(jn_collector_submit(c, id, 1, 64, 1, now - 1) == JN_EINVAL);
    int32_t pending = 0;
    int64_t deadline = 0;
    CHECK(jn_collector_status(c, &pending, &deadline) == JN_OK);
    std::vector<int64_t> ids(4096);
    int32_t got = 0;
    for (int guard = 0; guard < 200 && pending > 0; ++guard) {
      CHECK(jn_collector_poll(c, now + 1000000, ids.data(), (int)ids.size(), &got) == JN_OK);
      out += got;
      CHECK(jn_collector_status(c, &pending, &deadline) == JN_OK);
    }
    CHECK(pending == 0 && out == n + 1);
    jn_collector_destroy(c);
  }
  jn_collector* c = nullptr;
  CHECK(jn_collector_create(&c, 0, 1) == JN_EINVAL);
}

// ---------------------------------------------------------- backbone ---

struct Bb {
  std::vector<jn_layer> layers;
  jn_backbone bb{};
};

Bb make_backbone(int L, int d, int H, int Hkv, int f, bool glu, int causal, float theta) {
  Bb b;
  const int hd = d / H, kv = Hkv ? Hkv : H;
  for (int l = 0; l < L; ++l) {
    jn_layer x{};
    x.wqkv = dev((size_t)(H + 2 * kv) * hd * d * 2);
    x.wo = dev((size_t)d * d * 2);
    x.w_up = dev((size_t)f * d * 2);
    x.w_gate = glu ? dev((size_t)f * d * 2) : nullptr;
    x.w_down = dev((size_t)d * f * 2);
    x.g1 = dev(d * 2);
    x.g2 = dev(d * 2);
    b.layers.push_back(x);
  }
  b.bb.n_layers = L;
  b.bb.d = d;
  b.bb.n_heads = H;
  b.bb.ffn = f;
  b.bb.eps = 1e-6f;
  b.bb.n_kv_heads = Hkv;
  b.bb.layers = b.layers.data();
  b.bb.gf = dev(d * 2);
  b.bb.causal = causal;
  b.bb.rope_theta = theta;
  return b;
}

void run_backbone(jn_ctx* c, Bb& b, Packed& k) {
  size_t ws = 0;
  CHECK(jn_backbone_workspace_size(&b.bb, k.p.T, &ws) == JN_OK);
  void* w = dev(ws);
  void* hidden = dev((size_t)k.p.T * k.p.d * 2);
  CHECK(jn_backbone_forward(c, &b.bb, &k.p, hidden, w, ws) == JN_OK);
  CHECK(jn_backbone_forward(c, &b.bb, &k.p, hidden, w, ws - 1) == JN_ENOSPACE);
  std::free(w);
  g_allocs.pop_back();
  std::free(hidden);
  g_allocs.pop_back();
}

void check_backbones(jn_ctx* c) {
  Rng r(3);
  struct Case {
    int G, d, H, Hkv, f, glu, causal;
    float theta;
    int reqs, n, max_len, align;
  };
  const Case cases[] = {
      {2, 128, 4, 0, 512, 0, 0, 0.f, 1, 8, 32, 1},        // the tiny workload's shapes
      {3, 256, 4, 2, 384, 1, 1, 1e4f, 2, 6, 200, 16},     // causal, rope, grouped kv, GeGLU
      {2, 512, 2, 1, 1920, 1, 0, 500.f, 2, 40, 320, 1},   // multi-query, head width 256
      {4, 768, 12, 0, 3072, 0, 0, 0.f, 1, 32, 244, 1},    // 12 heads of 64
      {1, 512, 4, 0, 1408, 1, 0, 0.f, 1, 1, 3, 64},       // one short sample (split-K launches)
      {2, 384, 6, 0, 1408, 1, 0, 0.f, 2, 70, 320, 1},     // widths that are not multiples of 256
      {1, 2048, 8, 0, 8192, 1, 0, 0.f, 1, 40, 256, 1},    // long-K down projection: split row-split tail
  };
  for (const Case& cs : cases) {
    // the long-K case as 10,240 rows: 40 token tiles x 8 weight tiles, a
    // row-split tail of 2,048 rows
    Group g = cs.f >= 8192 ? fixed_group(cs.d, 40, 256) : make_group(r, cs.G, cs.d, cs.reqs, cs.n, cs.max_len, cs.align);
    Packed k = pack(c, g);
    const long long l0 = jn_fake_launches;
    Bb b = make_backbone(2, cs.d, cs.H, cs.Hkv, cs.f, cs.glu, cs.causal, cs.theta);
    run_backbone(c, b, k);
    // per layer: 2 norms, qkv, attention, o, geglu, down; + final norm; the
    // split tail adds a partial launch and a reduction to the down projection
    if (cs.f >= 8192) CHECK(jn_fake_launches - l0 == 2 * (2 + 1 + 1 + 2 + 1 + 3) + 1);
    CHECK(jn_ctx_set_trace(c, 1) == JN_OK);
    run_backbone(c, b, k);
    std::vector<jn_trace_entry> tr(4096);
    int32_t n = 0;
    CHECK(jn_ctx_trace_read(c, tr.data(), 8, &n) == JN_OK && n <= 8);
    CHECK(jn_ctx_set_trace(c, 0) == JN_OK);
    // unsupported shapes and bad variant fields enqueue nothing
    Bb bad = make_backbone(1, 4224, 33, 0, 512, 0, 0, 0.f);
    void* h = dev((size_t)k.p.T * 4224 * 2);
    CHECK(jn_backbone_forward(c, &bad.bb, &k.p, h, h, 16) == JN_EUNSUPPORTED);
    b.bb.n_kv_heads = 3;
    CHECK(jn_backbone_forward(c, &b.bb, &k.p, h, h, 16) != JN_OK);
  }
}

// ------------------------------------------------------------- heads ---

struct Heads {
  std::vector<std::vector<int32_t>> dims;
  std::vector<std::vector<const float*>> W, b;
  std::vector<std::vector<float*>> dW, db;
  std::vector<jn_head> h;
  std::vector<jn_head_io> io;
};

Heads make_heads(Rng& r, const Group& g, int d, int layers) {
  Heads H;
  const int G = (int)g.ten.size();
  H.dims.resize(G);
  H.W.resize(G);
  H.b.resize(G);
  H.dW.resize(G);
  H.db.resize(G);
  for (int t = 0; t < G; ++t) {
    int n = 0;
    for (const auto& q : g.req)
      if (q.tenant == t) n += q.n_samples;
    const int a = r.range(1, 32), ch = r.range(1, 10);
    H.dims[t].push_back(d);
    for (int l = 1; l < layers; ++l) H.dims[t].push_back(r.range(1, 300));
    H.dims[t].push_back(a * ch);
    for (int l = 0; l < layers; ++l) {
      const size_t in = H.dims[t][l], out = H.dims[t][l + 1];
      H.W[t].push_back((const float*)dev(4 * in * out));
      H.b[t].push_back((const float*)dev(4 * out));
      H.dW[t].push_back((float*)dev(4 * in * out));
      H.db[t].push_back((float*)dev(4 * out));
    }
    jn_head h{};
    h.n_layers = layers;
    h.action_dim = a;
    h.chunk = ch;
    H.h.push_back(h);
    jn_head_io io{};
    io.targets = (const float*)dev(4 * (size_t)n * a * ch);
    io.actions = (float*)dev(4 * (size_t)n * a * ch);
    io.loss = (float*)dev(4);
    H.io.push_back(io);
  }
  for (int t = 0; t < G; ++t) {
    H.h[t].dims = H.dims[t].data();
    H.h[t].W = H.W[t].data();
    H.h[t].b = H.b[t].data();
    H.io[t].dW = H.dW[t].data();
    H.io[t].db = H.db[t].data();
  }
  return H;
}

void check_heads(jn_ctx* c) {
  Rng r(4);
  for (int it = 0; it < 40; ++it) {
    const int d = 128 * r.range(1, 4);
    Group g = make_group(r, r.range(1, 6), d, 2, 40, 64, r.range(0, 1) ? 1 : 16);
    Packed k = pack(c, g);
    Heads H = make_heads(r, g, d, r.range(1, 4));
    const int G = (int)g.ten.size();
    size_t ws = 0;
    CHECK(jn_heads_workspace_size(&k.p, H.h.data(), G, &ws) == JN_OK);
    void* w = dev(ws);
    void* hidden = dev((size_t)k.p.T * d * 2);
    float* pooled = (float*)dev((size_t)4 * k.p.N * d);
    CHECK(jn_tenant_heads_fwd_bwd(c, &k.p, hidden, H.h.data(), H.io.data(), G, w, ws, pooled) == JN_OK);
    CHECK(jn_tenant_heads_fwd_bwd(c, &k.p, hidden, H.h.data(), H.io.data(), G, w, ws, nullptr) == JN_OK);
    CHECK(jn_tenant_heads_fwd_bwd(c, &k.p, hidden, H.h.data(), H.io.data(), G, w, ws - 1, pooled) == JN_ENOSPACE);
    CHECK(jn_tenant_heads_fwd_bwd_noalloc(c, &k.p, hidden, H.h.data(), H.io.data(), G, pooled) == JN_OK);
    if (G > 1) CHECK(jn_tenant_heads_fwd_bwd(c, &k.p, hidden, H.h.data(), H.io.data(), G - 1, w, ws, pooled) == JN_EINVAL);
    // unpack of the hidden rows, then of the same samples split differently
    std::vector<void*> outs;
    for (const auto& q : g.req) outs.push_back(dev((size_t)q.n_samples * q.max_len * d * 2));
    CHECK(jn_unpack(c, &k.p, g.req.data(), (int)g.req.size(), hidden, (size_t)d * 2, outs.data()) == JN_OK);
    CHECK(jn_unpack(c, &k.p, g.req.data(), (int)g.req.size(), hidden, 12, outs.data()) == JN_OK);
    if (g.req.size() > 1 && g.req[0].n_samples > 1) {
      std::vector<jn_request> moved(g.req);
      moved[0].n_samples -= 1;
      moved[1].n_samples += 1;
      CHECK(jn_unpack(c, &k.p, moved.data(), (int)moved.size(), hidden, (size_t)d * 2, outs.data()) == JN_ESHAPE);
    }
  }
}

// ------------------------------------------------------------ experts ---

void check_experts(jn_ctx* c, bool flow, bool long_prefix = false) {
  Rng r(flow ? 6 : 5);
  const int dp = 128, d = 256, H = 4, f = 512, L = 2, chunk = 10, dt = 64;
  // long prefixes: tenants with over 9K prefix rows, whose key/value weight
  // gradients run split into K ranges
  Group g = long_prefix ? long_group(dp, 3, 8, 1500) : make_group(r, 3, dp, 2, 4, 40, 16);
  Packed k = pack(c, g);
  const int G = 3;
  std::vector<int32_t> ns(G);
  std::vector<int64_t> rows(G);
  CHECK(jn_pack_tenant_sizes(g.req.data(), (int)g.req.size(), g.ten.data(), G, &g.opts, ns.data(), rows.data()) ==
        JN_OK);
  if (long_prefix) {
    int64_t most = 0;
    for (int t = 0; t < G; ++t) most = std::max(most, rows[t]);
    CHECK(most >= 9216);  // at least one tenant's prefix gradient is split
  }
  std::vector<jn_expert> ex(G);
  std::vector<jn_expert_io> io(G);
  std::vector<std::vector<jn_expert_layer>> xl(G);
  std::vector<std::vector<jn_expert_layer_grads>> gl(G);
  for (int t = 0; t < G; ++t) {
    const int a = r.range(1, 32);
    for (int l = 0; l < L; ++l) {
      jn_expert_layer x{};
      x.wqkv_s = dev((size_t)3 * d * d * 2);
      x.wo_s = dev((size_t)d * d * 2);
      x.wq_c = dev((size_t)d * d * 2);
      x.wkv_c = dev((size_t)2 * d * dp * 2);
      x.wo_c = dev((size_t)d * d * 2);
      x.w_up = dev((size_t)f * d * 2);
      x.w_down = dev((size_t)d * f * 2);
      x.g1 = dev(d * 2);
      x.g2 = dev(d * 2);
      x.g3 = dev(d * 2);
      xl[t].push_back(x);
      jn_expert_layer_grads y{};
      y.wqkv_s = (float*)dev((size_t)3 * d * d * 4);
      y.wo_s = (float*)dev((size_t)d * d * 4);
      y.wq_c = (float*)dev((size_t)d * d * 4);
      y.wkv_c = (float*)dev((size_t)2 * d * dp * 4);
      y.wo_c = (float*)dev((size_t)d * d * 4);
      y.w_up = (float*)dev((size_t)f * d * 4);
      y.w_down = (float*)dev((size_t)d * f * 4);
      y.g1 = (float*)dev(d * 4);
      y.g2 = (float*)dev(d * 4);
      y.g3 = (float*)dev(d * 4);
      gl[t].push_back(y);
    }
    jn_expert& e = ex[t];
    e.n_layers = L;
    e.d = d;
    e.n_heads = H;
    e.ffn = f;
    e.action_dim = a;
    e.chunk = chunk;
    e.d_prefix = dp;
    e.eps = 1e-6f;
    e.w_in = dev((size_t)d * a * 2);
    e.w_out = dev((size_t)a * d * 2);
    e.gf = dev(d * 2);
    e.w_time = flow ? dev((size_t)d * dt * 2) : nullptr;
    e.d_time = flow ? dt : 0;
    jn_expert_io& o = io[t];
    o.n_samples = ns[t];
    o.prefix_rows = rows[t];
    const size_t act = (size_t)ns[t] * chunk * a * 4;
    o.noisy = (const float*)dev(act);
    o.targets = (const float*)dev(act);
    o.pred = (float*)dev(act);
    o.loss = (float*)dev(4);
    o.dw_in = (float*)dev((size_t)d * a * 4);
    o.dw_out = (float*)dev((size_t)a * d * 4);
    o.dgf = (float*)dev(d * 4);
    o.flow_t = flow ? (const float*)dev(4 * (size_t)ns[t]) : nullptr;
    o.dw_time = flow ? (float*)dev((size_t)d * dt * 4) : nullptr;
  }
  for (int t = 0; t < G; ++t) {
    ex[t].layers = xl[t].data();
    io[t].layers = gl[t].data();
  }
  size_t ws = 0;
  CHECK(jn_experts_workspace_size(&k.p, ex.data(), io.data(), G, &ws) == JN_OK);
  void* w = dev(ws);
  void* hidden = dev((size_t)k.p.T * dp * 2);
  CHECK(jn_tenant_experts_fwd_bwd(c, &k.p, hidden, ex.data(), io.data(), G, w, ws) == JN_OK);
  // the materialised-transpose path of the gradient GEMMs plans within the same workspace
  CHECK(jn_ctx_set_option(c, JN_OPT_EXPERT_TRANSPOSES, 1) == JN_OK);
  CHECK(jn_tenant_experts_fwd_bwd(c, &k.p, hidden, ex.data(), io.data(), G, w, ws) == JN_OK);
  CHECK(jn_ctx_set_option(c, JN_OPT_EXPERT_TRANSPOSES, 0) == JN_OK);
  CHECK(jn_ctx_set_option(c, JN_OPT_EXPERT_TRANSPOSES, 2) == JN_EINVAL);
  CHECK(jn_ctx_set_option(c, 99, 0) == JN_EINVAL);
  CHECK(jn_ctx_set_option(nullptr, JN_OPT_EXPERT_TRANSPOSES, 0) == JN_EINVAL);
  CHECK(jn_tenant_experts_fwd_bwd(c, &k.p, hidden, ex.data(), io.data(), G, w, ws - 1) == JN_ENOSPACE);
  ex[0].chunk = 65;
  CHECK(jn_tenant_experts_fwd_bwd(c, &k.p, hidden, ex.data(), io.data(), G, w, ws) == JN_EUNSUPPORTED);
  ex[0].chunk = chunk;
  io[1].n_samples += 1;
  CHECK(jn_tenant_experts_fwd_bwd(c, &k.p, hidden, ex.data(), io.data(), G, w, ws) != JN_OK);
}

// ---------------------------------------------------------- optimizer ---

void check_adamw(jn_ctx* c) {
  Rng r(7);
  const int G = 3;
  std::vector<jn_adamw_tenant> t(G);
  std::vector<std::vector<float*>> p(G), m(G), v(G);
  std::vector<std::vector<const float*>> gr(G);
  std::vector<std::vector<int64_t>> n(G);
  std::vector<std::vector<void*>> b16(G);
  for (int k = 0; k < G; ++k) {
    const int nt = r.range(1, 6);
    for (int i = 0; i < nt; ++i) {
      const int64_t e = r.range(1, 70001);
      n[k].push_back(e);
      p[k].push_back((float*)dev(4 * e));
      gr[k].push_back((const float*)dev(4 * e));
      m[k].push_back((float*)dev(4 * e));
      v[k].push_back((float*)dev(4 * e));
      b16[k].push_back(i % 2 ? dev(2 * e) : nullptr);
    }
    t[k] = jn_adamw_tenant{1e-3f, 0.9f, 0.999f, 1e-8f, 0.01f, nt, 1 + k, p[k].data(), gr[k].data(), m[k].data(),
                           v[k].data(), n[k].data(), b16[k].data()};
  }
  size_t ws = 0;
  CHECK(jn_adamw_workspace_size(t.data(), G, &ws) == JN_OK);
  void* w = dev(ws);
  CHECK(jn_tenant_adamw_step(c, t.data(), G, w, ws) == JN_OK);
  CHECK(jn_tenant_adamw_step(c, t.data(), G, w, ws - 1) == JN_ENOSPACE);
  t[1].step = 0;
  CHECK(jn_tenant_adamw_step(c, t.data(), G, w, ws) == JN_EINVAL);
}

// ---------------------------------------------------------- inference ---

void check_infer(jn_ctx* c, void* stream) {
  Rng r(8);
  const int d = 256;
  Group g = make_group(r, 3, d, 2, 4, 60, 1);
  Heads H = make_heads(r, g, d, 2);
  Bb b = make_backbone(2, d, 4, 0, 512, 1, 0, 0.f);
  const int G = 3;
  size_t ws = 0;
  CHECK(jn_infer_workspace_size(g.req.data(), (int)g.req.size(), g.ten.data(), G, &g.opts, &b.bb, H.h.data(), &ws) ==
        JN_OK);
  void* w = dev(ws);
  std::vector<float*> acts;
  for (int t = 0; t < G; ++t) acts.push_back(H.io[t].actions);
  jn_infer_plan* pl = nullptr;
  CHECK(jn_infer_plan_create(c, g.req.data(), (int)g.req.size(), g.ten.data(), G, &g.opts, &b.bb, H.h.data(),
                             acts.data(), w, ws - 1, &pl) == JN_ENOSPACE);
  CHECK(jn_infer_plan_create(c, g.req.data(), (int)g.req.size(), g.ten.data(), G, &g.opts, &b.bb, H.h.data(),
                             acts.data(), w, ws, &pl) == JN_OK);
  CHECK(jn_infer_plan_replay(c, pl) == JN_EINVAL);   // nothing captured yet
  CHECK(jn_infer_plan_launch(c, pl) == JN_OK);
  CHECK(jn_ctx_set_stream(c, stream) == JN_OK);
  CHECK(jn_infer_plan_capture(c, pl) == JN_OK);
  const long long before = jn_fake_graph_launches;
  CHECK(jn_infer_plan_replay(c, pl) == JN_OK && jn_fake_graph_launches == before + 1);
  jn_packed pk{};
  void* hidden = nullptr;
  CHECK(jn_infer_plan_packed(pl, &pk, &hidden) == JN_OK && hidden != nullptr);
  jn_infer_plan_destroy(pl);
  CHECK(jn_ctx_set_stream(c, nullptr) == JN_OK);
}

}  // namespace

int main() {
  check_plans();
  check_collector();
  jn_ctx* c = nullptr;
  CHECK(jn_ctx_create(&c, nullptr) == JN_OK);
  check_backbones(c);
  check_heads(c);
  check_experts(c, false);
  check_experts(c, true);
  check_experts(c, false, true);
  check_adamw(c);
  int stream_token = 0;
  check_infer(c, &stream_token);
  CHECK(std::strlen(jn_last_error(c)) > 0);
  jn_ctx_destroy(c);
  for (void* p : g_allocs) std::free(p);
  std::printf("host checks ok: %d checks, %lld launches\n", g_checks, jn_fake_launches);
  return 0;
}
