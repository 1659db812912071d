// Host side of the C ABI: validation, the pack plan, workspace carving,
// pinned staging of small tables, and launch sequencing on the context stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <deque>
#include <functional>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "jn_internal.h"

using namespace jnx;

// ------------------------------------------------- library-owned scratch ---

// Workspace of jn_tenant_heads_fwd_bwd_noalloc: one array per GPU, held
// until the process ends.  Host code never uses its name as an address (on
// the host it is a stand-in symbol); the device address comes from
// hipGetSymbolAddress, once per device, and is kept per device.
namespace {
constexpr size_t kHeadsScratchBytes = size_t(JN_HEADS_SCRATCH_BYTES);
constexpr size_t kFixedStageBytes = size_t(1) << 20;
constexpr int kMaxDevices = 64;
}  // namespace

static __device__ __align__(256) char scratch[kHeadsScratchBytes];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
bool g_scratch_done[kMaxDevices] = {};

// Device address of `scratch` on `dev` (which must be the current device);
// nullptr if the runtime could not resolve it.
void* scratch_address(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_done[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) {
      (void)hipGetLastError();
      ptr = nullptr;
    }
    g_scratch_ptr[dev] = ptr;
    g_scratch_done[dev] = true;
  }
  return g_scratch_ptr[dev];
}
}  // namespace

// --------------------------------------------------------------- context ---

namespace {
constexpr int kSlots = 8;      // staging slots at context creation
constexpr int kMaxSlots = 64;  // the ring grows to this many before the host waits
struct StageSlot {
  void* host = nullptr;
  size_t cap = 0;
  hipEvent_t ev = nullptr;
  bool pending = false;
};
}  // namespace

namespace {
struct TraceRec {
  int32_t op, M, N, K;
  hipEvent_t start, stop;
};
}  // namespace

struct jn_ctx {
  hipStream_t stream = nullptr;
  int device = 0;
  std::string err;
  std::vector<StageSlot> slots = std::vector<StageSlot>(kSlots);
  int next = 0;
  // launch trace (measurement only): a pair of timing events around every
  // kernel launch while enabled
  bool trace = false;
  std::vector<TraceRec> recs;
  std::vector<hipEvent_t> pool;
  size_t pool_used = 0;
  // allocation-free entry points: the device's library-owned scratch array
  // (resolved at creation) and a pinned staging buffer of fixed size for
  // their tables, allocated at creation and never grown
  void* scratch = nullptr;
  void* fixed_host = nullptr;
  hipEvent_t fixed_ev = nullptr;
  bool fixed_pending = false;
  // JN_OPT_EXPERT_TRANSPOSES
  bool expert_transposes = false;
};

namespace {

jn_status fail(jn_ctx* c, jn_status code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c) c->err = buf;
  return code;
}

jn_status hip_fail(jn_ctx* c, hipError_t e, const char* what) {
  return fail(c, JN_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define JN_HIP(ctx, call, what)                         \
  do {                                                  \
    hipError_t _e = (call);                             \
    if (_e != hipSuccess) return hip_fail(ctx, _e, what); \
  } while (0)

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

hipEvent_t trace_event(jn_ctx* c) {
  if (c->pool_used == c->pool.size()) {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    c->pool.push_back(e);
  }
  return c->pool[c->pool_used++];
}

// Enqueue one kernel launch; with tracing on, bracket it with timing events.
template <typename F>
hipError_t traced(jn_ctx* c, int32_t op, int64_t M, int64_t N, int64_t K, F&& launch) {
  if (!c->trace) return launch();
  hipEvent_t a = trace_event(c), b = trace_event(c);
  if (!a || !b) return hipErrorOutOfMemory;
  hipError_t e = hipEventRecord(a, c->stream);
  if (e != hipSuccess) return e;
  e = launch();
  if (e != hipSuccess) return e;
  e = hipEventRecord(b, c->stream);
  if (e != hipSuccess) return e;
  c->recs.push_back(TraceRec{op, (int32_t)M, (int32_t)N, (int32_t)K, a, b});
  return hipSuccess;
}

#define JN_TRACED(ctx, op, M, N, K, call, what) \
  JN_HIP(ctx, traced(ctx, op, M, N, K, [&]() { return (call); }), what)

// Stage `bytes` of host data in pinned memory and copy it to `dst` on the
// context stream.  Slots are reused round-robin; a slot is rewritten only
// after the copy that last read it has completed.  When the next slot's copy
// is still in flight the ring grows by a slot instead (up to kMaxSlots), so
// the host does not wait on the device while the device runs behind by fewer
// than kMaxSlots uploads.
jn_status stage_copy(jn_ctx* c, void* dst, const void* src, size_t bytes) {
  if (bytes == 0) return JN_OK;
  if (c->slots[c->next].pending && hipEventQuery(c->slots[c->next].ev) == hipErrorNotReady &&
      c->slots.size() < (size_t)kMaxSlots) {
    StageSlot fresh;
    JN_HIP(c, hipEventCreateWithFlags(&fresh.ev, hipEventDisableTiming), "hipEventCreate(staging)");
    c->slots.insert(c->slots.begin() + c->next, fresh);
  }
  StageSlot& s = c->slots[c->next];
  c->next = (c->next + 1) % (int)c->slots.size();
  if (s.pending) {
    JN_HIP(c, hipEventSynchronize(s.ev), "hipEventSynchronize(staging)");
    s.pending = false;
  }
  if (s.cap < bytes) {
    if (s.host) JN_HIP(c, hipHostFree(s.host), "hipHostFree");
    s.host = nullptr;
    s.cap = 0;
    size_t cap = align_up(std::max<size_t>(bytes, 1 << 16), 1 << 16);
    JN_HIP(c, hipHostMalloc(&s.host, cap, hipHostMallocDefault), "hipHostMalloc(staging)");
    s.cap = cap;
  }
  std::memcpy(s.host, src, bytes);
  JN_HIP(c, hipMemcpyAsync(dst, s.host, bytes, hipMemcpyHostToDevice, c->stream), "hipMemcpyAsync(H2D)");
  JN_HIP(c, hipEventRecord(s.ev, c->stream), "hipEventRecord(staging)");
  s.pending = true;
  return JN_OK;
}

// Stage a table through the context's fixed pinned buffer (the
// allocation-free entry points): never allocates; JN_ENOSPACE if the table
// does not fit.
jn_status stage_copy_fixed(jn_ctx* c, void* dst, const void* src, size_t bytes) {
  if (bytes == 0) return JN_OK;
  if (bytes > kFixedStageBytes)
    return fail(c, JN_ENOSPACE, "tables of %zu B exceed the %zu B fixed staging buffer", bytes, kFixedStageBytes);
  if (c->fixed_pending) {
    JN_HIP(c, hipEventSynchronize(c->fixed_ev), "hipEventSynchronize(fixed staging)");
    c->fixed_pending = false;
  }
  std::memcpy(c->fixed_host, src, bytes);
  JN_HIP(c, hipMemcpyAsync(dst, c->fixed_host, bytes, hipMemcpyHostToDevice, c->stream), "hipMemcpyAsync(H2D)");
  JN_HIP(c, hipEventRecord(c->fixed_ev, c->stream), "hipEventRecord(fixed staging)");
  c->fixed_pending = true;
  return JN_OK;
}

// ------------------------------------------------------------------ plan ---

struct MapLayout {
  size_t seqlens, cu, sreq, sloc, sten, toff, tperm, trank, tsamp, tpos, reqtab, total;
};

MapLayout map_layout(int64_t N, int64_t T, int64_t G, int64_t R) {
  MapLayout m{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align_up(o + bytes, 256);
    return at;
  };
  m.seqlens = take(4 * N);
  m.cu = take(4 * (N + 1));
  m.sreq = take(4 * N);
  m.sloc = take(4 * N);
  m.sten = take(4 * N);
  m.toff = take(4 * (G + 1));
  m.tperm = take(4 * N);
  m.trank = take(4 * N);
  m.tsamp = take(4 * T);
  m.tpos = take(4 * T);
  m.reqtab = take(sizeof(ReqEntry) * R);
  m.total = o;
  return m;
}

struct Plan {
  int32_t N = 0, T = 0, max_seqlen = 0, max_rows = 0, max_req_len = 0;
  std::vector<int32_t> seqlens, cu, sreq, sloc, sten, toff, tperm, trank;
  std::vector<int32_t> req_first;
};

// Validates the request / tenant tables and computes every N- and G-sized
// map.  Arrival order = request order, samples in order; tenant order is a
// stable counting sort by tenant slot.
jn_status make_plan(jn_ctx* c, const jn_request* req, int32_t R, const jn_tenant* ten, int32_t G,
                    const jn_pack_opts* o, Plan* p) {
  if (!req || !ten || !o || !p) return fail(c, JN_EINVAL, "null argument");
  if (R < 1) return fail(c, JN_EINVAL, "need at least one request (R=%d)", R);
  if (G < 1) return fail(c, JN_EINVAL, "need at least one tenant (G=%d)", G);
  if (o->align < 1 || o->align > 4096) return fail(c, JN_EINVAL, "align %d outside [1, 4096]", o->align);
  if (o->d_model < 1) return fail(c, JN_EINVAL, "d_model %d < 1", o->d_model);
  for (int32_t g = 0; g < G; ++g) {
    if (ten[g].prefix_sig != ten[0].prefix_sig)
      return fail(c, JN_EINCOMPAT, "tenant %d has a different shared-prefix signature", g);
    if (ten[g].d_model != o->d_model)
      return fail(c, JN_EINCOMPAT, "tenant %d expects width %d, backbone has %d", g, ten[g].d_model,
                  o->d_model);
  }
  int64_t N = 0;
  for (int32_t r = 0; r < R; ++r) {
    if (req[r].tenant < 0 || req[r].tenant >= G)
      return fail(c, JN_ESHAPE, "request %d names tenant %d outside the table of %d", r, req[r].tenant, G);
    if (req[r].n_samples < 1) return fail(c, JN_ESHAPE, "request %d has no samples", r);
    if (req[r].max_len < 1) return fail(c, JN_ESHAPE, "request %d has max_len %d", r, req[r].max_len);
    if (!req[r].embeds || !req[r].lengths) return fail(c, JN_EINVAL, "request %d has a null pointer", r);
    N += req[r].n_samples;
  }
  if (N >= (1ll << 30)) return fail(c, JN_ESHAPE, "too many samples");
  p->N = (int32_t)N;
  p->seqlens.resize(N);
  p->cu.resize(N + 1);
  p->sreq.resize(N);
  p->sloc.resize(N);
  p->sten.resize(N);
  p->req_first.resize(R);
  int64_t i = 0, T = 0;
  int32_t mx = 0, mreq = 0;
  p->cu[0] = 0;
  for (int32_t r = 0; r < R; ++r) {
    p->req_first[r] = (int32_t)i;
    mreq = std::max(mreq, req[r].max_len);
    for (int32_t s = 0; s < req[r].n_samples; ++s, ++i) {
      int32_t L = req[r].lengths[s];
      if (L < 1 || L > req[r].max_len)
        return fail(c, JN_ESHAPE, "request %d sample %d: length %d outside [1, %d]", r, s, L, req[r].max_len);
      int64_t rows = (int64_t)(L + o->align - 1) / o->align * o->align;
      T += rows;
      if (T >= (1ll << 31) - 1) return fail(c, JN_ESHAPE, "packed batch overflows int32 row indices");
      p->seqlens[i] = L;
      p->cu[i + 1] = (int32_t)T;
      p->sreq[i] = r;
      p->sloc[i] = s;
      p->sten[i] = req[r].tenant;
      mx = std::max(mx, L);
    }
  }
  p->T = (int32_t)T;
  p->max_seqlen = mx;
  p->max_rows = (int32_t)((int64_t)(mx + o->align - 1) / o->align * o->align);
  p->max_req_len = mreq;
  p->toff.assign(G + 1, 0);
  for (int64_t k = 0; k < N; ++k) p->toff[p->sten[k] + 1]++;
  for (int32_t g = 0; g < G; ++g) {
    if (p->toff[g + 1] == 0) return fail(c, JN_ESHAPE, "tenant %d has no samples in this group", g);
    p->toff[g + 1] += p->toff[g];
  }
  p->tperm.resize(N);
  p->trank.resize(N);
  std::vector<int32_t> fill(p->toff.begin(), p->toff.end() - 1);
  for (int64_t k = 0; k < N; ++k) {
    int32_t pos = fill[p->sten[k]]++;
    p->tperm[pos] = (int32_t)k;
    p->trank[k] = pos;
  }
  return JN_OK;
}

void fill_packed(jn_packed* out, char* base, const MapLayout& m, const Plan& p, int32_t R, int32_t G,
                 const jn_pack_opts* o) {
  std::memset(out, 0, sizeof(*out));
  out->R = R;
  out->G = G;
  out->N = p.N;
  out->T = p.T;
  out->d = o->d_model;
  out->max_seqlen = p.max_seqlen;
  out->align = o->align;
  for (int32_t g = 0; g < G; ++g) out->max_tenant_n = std::max(out->max_tenant_n, p.toff[g + 1] - p.toff[g]);
  out->seqlens = (int32_t*)(base + m.seqlens);
  out->cu_seqlens = (int32_t*)(base + m.cu);
  out->sample_request = (int32_t*)(base + m.sreq);
  out->sample_local = (int32_t*)(base + m.sloc);
  out->sample_tenant = (int32_t*)(base + m.sten);
  out->tenant_sample_off = (int32_t*)(base + m.toff);
  out->tenant_perm = (int32_t*)(base + m.tperm);
  out->sample_tenant_rank = (int32_t*)(base + m.trank);
  out->token_sample = (int32_t*)(base + m.tsamp);
  out->token_pos = (int32_t*)(base + m.tpos);
  out->req_table = base + m.reqtab;
}

// Host image of the maps region [0, m.tsamp) (the N/G-sized arrays).
std::vector<char> host_head_image(const MapLayout& m, const Plan& p) {
  std::vector<char> img(m.tsamp, 0);
  auto put = [&](size_t off, const std::vector<int32_t>& v) {
    if (!v.empty()) std::memcpy(img.data() + off, v.data(), 4 * v.size());
  };
  put(m.seqlens, p.seqlens);
  put(m.cu, p.cu);
  put(m.sreq, p.sreq);
  put(m.sloc, p.sloc);
  put(m.sten, p.sten);
  put(m.toff, p.toff);
  put(m.tperm, p.tperm);
  put(m.trank, p.trank);
  return img;
}

// Signature of the request shapes a physical batch was planned from: FNV-1a
// over R and every request's (n_samples, max_len).  jn_unpack compares it
// with the requests it is given, because the unpack kernel indexes each
// request's buffer with the pack-time sample positions.
int32_t request_signature(const jn_request* req, int32_t R) {
  uint32_t h = 2166136261u;
  auto mix = [&](uint32_t v) {
    for (int b = 0; b < 4; ++b) {
      h ^= (v >> (8 * b)) & 0xffu;
      h *= 16777619u;
    }
  };
  mix((uint32_t)R);
  for (int32_t r = 0; r < R; ++r) {
    mix((uint32_t)req[r].n_samples);
    mix((uint32_t)req[r].max_len);
  }
  return (int32_t)h;
}

bool valid_packed(const jn_packed* p) {
  return p && p->N > 0 && p->T > 0 && p->G > 0 && p->R > 0 && p->d > 0 && p->seqlens && p->cu_seqlens &&
         p->sample_request && p->sample_local && p->tenant_sample_off && p->sample_tenant_rank &&
         p->req_table && p->max_tenant_n >= 0 && p->max_tenant_n <= p->N;
}

// Row bound of a per-tenant launch: the largest tenant's samples when the
// packing recorded it, else every sample.
int64_t tenant_rows_bound(const jn_packed* p) { return p->max_tenant_n > 0 ? p->max_tenant_n : p->N; }

}  // namespace

// ------------------------------------------------------------------ ABI ----

extern "C" {

jn_status jn_ctx_create(jn_ctx** out, void* hip_stream) {
  if (!out) return JN_EINVAL;
  *out = nullptr;
  jn_ctx* c = new (std::nothrow) jn_ctx();
  if (!c) return JN_EINVAL;
  c->stream = (hipStream_t)hip_stream;
  if (hipGetDevice(&c->device) != hipSuccess) {
    delete c;
    return JN_EHIP;
  }
  for (auto& s : c->slots) {
    if (hipEventCreateWithFlags(&s.ev, hipEventDisableTiming) != hipSuccess) {
      jn_ctx_destroy(c);
      return JN_EHIP;
    }
  }
  if (hipEventCreateWithFlags(&c->fixed_ev, hipEventDisableTiming) != hipSuccess ||
      hipHostMalloc(&c->fixed_host, kFixedStageBytes, hipHostMallocDefault) != hipSuccess) {
    c->fixed_host = nullptr;
    jn_ctx_destroy(c);
    return JN_EHIP;
  }
  c->scratch = scratch_address(c->device);
  *out = c;
  return JN_OK;
}

void jn_ctx_destroy(jn_ctx* c) {
  if (!c) return;
  for (auto& s : c->slots) {
    if (s.pending) hipEventSynchronize(s.ev);
    if (s.host) hipHostFree(s.host);
    if (s.ev) hipEventDestroy(s.ev);
  }
  if (c->fixed_pending) hipEventSynchronize(c->fixed_ev);
  if (c->fixed_host) hipHostFree(c->fixed_host);
  if (c->fixed_ev) hipEventDestroy(c->fixed_ev);
  if (!c->recs.empty()) hipEventSynchronize(c->recs.back().stop);
  for (hipEvent_t e : c->pool) hipEventDestroy(e);
  delete c;
}

jn_status jn_ctx_set_stream(jn_ctx* c, void* hip_stream) {
  if (!c) return JN_EINVAL;
  c->stream = (hipStream_t)hip_stream;
  return JN_OK;
}

const char* jn_last_error(const jn_ctx* c) { return c ? c->err.c_str() : "null context"; }

jn_status jn_ctx_set_trace(jn_ctx* c, int32_t enable) {
  if (!c) return JN_EINVAL;
  c->trace = enable != 0;
  c->recs.clear();
  c->pool_used = 0;
  return JN_OK;
}

jn_status jn_ctx_set_option(jn_ctx* c, int32_t option, int32_t value) {
  if (!c) return JN_EINVAL;
  if (value != 0 && value != 1) return fail(c, JN_EINVAL, "option %d: value %d is not 0 or 1", option, value);
  switch (option) {
    case JN_OPT_EXPERT_TRANSPOSES: c->expert_transposes = value != 0; return JN_OK;
    default: return fail(c, JN_EINVAL, "unknown option %d", option);
  }
}

jn_status jn_ctx_trace_read(jn_ctx* c, jn_trace_entry* out, int32_t cap, int32_t* n) {
  if (!c || !n || (cap > 0 && !out)) return JN_EINVAL;
  *n = 0;
  if (!c->recs.empty()) JN_HIP(c, hipEventSynchronize(c->recs.back().stop), "hipEventSynchronize(trace)");
  int32_t k = 0;
  for (const TraceRec& r : c->recs) {
    if (k >= cap) break;
    float ms = 0.f;
    JN_HIP(c, hipEventElapsedTime(&ms, r.start, r.stop), "hipEventElapsedTime");
    out[k] = jn_trace_entry{r.op, r.M, r.N, r.K, ms, 0};
    ++k;
  }
  *n = k;
  c->recs.clear();
  c->pool_used = 0;
  return JN_OK;
}

jn_status jn_pack_plan(const jn_request* req, int32_t R, const jn_tenant* ten, int32_t G,
                       const jn_pack_opts* o, jn_pack_sizes* out) {
  if (!out) return JN_EINVAL;
  Plan p;
  jn_status st = make_plan(nullptr, req, R, ten, G, o, &p);
  if (st != JN_OK) return st;
  MapLayout m = map_layout(p.N, p.T, G, R);
  std::memset(out, 0, sizeof(*out));
  out->N = p.N;
  out->T = p.T;
  out->max_seqlen = p.max_seqlen;
  out->map_bytes = (int64_t)m.total;
  out->token_bytes = (int64_t)p.T * o->d_model * 2;
  return JN_OK;
}

jn_status jn_pack_maps_host(const jn_request* req, int32_t R, const jn_tenant* ten, int32_t G,
                            const jn_pack_opts* o, void* host_maps, size_t map_bytes, jn_packed* out) {
  if (!host_maps || !out) return JN_EINVAL;
  Plan p;
  jn_status st = make_plan(nullptr, req, R, ten, G, o, &p);
  if (st != JN_OK) return st;
  MapLayout m = map_layout(p.N, p.T, G, R);
  if (map_bytes < m.total) return JN_ENOSPACE;
  std::vector<char> img = host_head_image(m, p);
  char* base = (char*)host_maps;
  std::memset(base, 0, m.total);
  std::memcpy(base, img.data(), img.size());
  int32_t* ts = (int32_t*)(base + m.tsamp);
  int32_t* tp = (int32_t*)(base + m.tpos);
  for (int32_t i = 0; i < p.N; ++i) {
    for (int32_t t = p.cu[i]; t < p.cu[i + 1]; ++t) {
      int32_t j = t - p.cu[i];
      ts[t] = j < p.seqlens[i] ? i : -1;
      tp[t] = j < p.seqlens[i] ? j : -1;
    }
  }
  ReqEntry* rt = (ReqEntry*)(base + m.reqtab);
  for (int32_t r = 0; r < R; ++r) rt[r] = ReqEntry{req[r].embeds, nullptr, req[r].max_len, req[r].n_samples, p.req_first[r], 0};
  fill_packed(out, base, m, p, R, G, o);
  out->req_sig = request_signature(req, R);
  return JN_OK;
}

jn_status jn_pack_group(jn_ctx* c, const jn_request* req, int32_t R, const jn_tenant* ten, int32_t G,
                        const jn_pack_opts* o, void* maps, size_t map_bytes, void* tokens,
                        size_t token_bytes, jn_packed* out) {
  if (!c) return JN_EINVAL;
  if (!maps || !tokens || !out) return fail(c, JN_EINVAL, "null output buffer");
  Plan p;
  jn_status st = make_plan(c, req, R, ten, G, o, &p);
  if (st != JN_OK) return st;
  MapLayout m = map_layout(p.N, p.T, G, R);
  if (map_bytes < m.total) return fail(c, JN_ENOSPACE, "map buffer %zu B < %zu B", map_bytes, m.total);
  size_t need_tok = (size_t)p.T * o->d_model * 2;
  if (token_bytes < need_tok) return fail(c, JN_ENOSPACE, "token buffer %zu B < %zu B", token_bytes, need_tok);
  if (o->d_model % 8 != 0) return fail(c, JN_EUNSUPPORTED, "d_model %d not a multiple of 8", o->d_model);
  for (int32_t r = 0; r < R; ++r)
    if (((uintptr_t)req[r].embeds) % 16 != 0) return fail(c, JN_EUNSUPPORTED, "request %d embeds not 16-byte aligned", r);
  if (((uintptr_t)tokens) % 16 != 0) return fail(c, JN_EUNSUPPORTED, "token buffer not 16-byte aligned");

  std::vector<char> img = host_head_image(m, p);
  std::vector<ReqEntry> rt(R);
  for (int32_t r = 0; r < R; ++r) rt[r] = ReqEntry{req[r].embeds, nullptr, req[r].max_len, req[r].n_samples, p.req_first[r], 0};
  char* base = (char*)maps;
  st = stage_copy(c, base, img.data(), img.size());
  if (st != JN_OK) return st;
  st = stage_copy(c, base + m.reqtab, rt.data(), sizeof(ReqEntry) * R);
  if (st != JN_OK) return st;
  jn_packed tmp;
  fill_packed(&tmp, base, m, p, R, G, o);
  tmp.req_sig = request_signature(req, R);
  tmp.tokens = tokens;
  JN_TRACED(c, JN_OP_PACK, p.T, o->d_model, 0,
            launch_pack(c->stream, (const ReqEntry*)tmp.req_table, tmp.sample_request, tmp.sample_local,
                        tmp.seqlens, tmp.cu_seqlens, p.N, o->d_model, o->align, p.max_rows, tokens,
                        tmp.token_sample, tmp.token_pos),
            "pack kernel");
  *out = tmp;
  return JN_OK;
}

// -------------------------------------------------------------- backbone ---

namespace {

struct BbLayout {
  size_t x, h, qkv, att, mid, split, split_bytes, total;
};

BbLayout bb_layout(const jn_backbone* bb, int64_t T) {
  BbLayout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align_up(o + bytes, 256);
    return at;
  };
  int64_t d = bb->d, f = bb->ffn;
  L.x = take(4 * T * d);
  L.h = take(2 * T * d);
  L.qkv = take(2 * T * 3 * d);
  L.att = take(2 * T * d);
  L.mid = take(2 * T * f);
  // fp32 partials of the split-K launches (short batches only)
  const bool glu = bb->layers && bb->layers[0].w_gate != nullptr;
  const int64_t kvh = bb->n_kv_heads ? bb->n_kv_heads : bb->n_heads;
  const int64_t nqkv = (bb->n_heads + 2 * kvh) * (d / bb->n_heads);
  size_t sb = std::max(gemm_split_bytes(EPI_BF16, (int32_t)T, (int32_t)nqkv, (int32_t)d),
                       gemm_split_bytes(EPI_RESID_F32, (int32_t)T, (int32_t)d, (int32_t)d));
  sb = std::max(sb, gemm_split_bytes(EPI_RESID_F32, (int32_t)T, (int32_t)d, (int32_t)f));
  if (!glu) sb = std::max(sb, gemm_split_bytes(EPI_GELU_BF16, (int32_t)T, (int32_t)f, (int32_t)d));
  L.split_bytes = sb;
  L.split = take(sb);
  L.total = o;
  return L;
}

jn_status check_backbone(jn_ctx* c, const jn_backbone* bb) {
  if (!bb || !bb->layers || !bb->gf) return fail(c, JN_EINVAL, "null backbone");
  if (bb->n_layers < 1 || bb->d < 1 || bb->n_heads < 1 || bb->ffn < 1)
    return fail(c, JN_EINVAL, "backbone sizes must be positive");
  if (bb->d % bb->n_heads != 0) return fail(c, JN_EINVAL, "d %% n_heads != 0");
  int hd = bb->d / bb->n_heads;
  if (hd != 32 && hd != 64 && hd != 128 && hd != 256)
    return fail(c, JN_EUNSUPPORTED, "head dim %d not in {32,64,128,256}", hd);
  if (bb->d % 128 != 0 || bb->d > 4096)
    return fail(c, JN_EUNSUPPORTED, "d %d not a multiple of 128 in [128, 4096]", bb->d);
  if (bb->ffn % 128 != 0) return fail(c, JN_EUNSUPPORTED, "ffn %d not a multiple of 128", bb->ffn);
  if (!(bb->eps > 0.f)) return fail(c, JN_EINVAL, "eps must be > 0");
  const int kv = bb->n_kv_heads ? bb->n_kv_heads : bb->n_heads;
  if (kv < 1 || bb->n_heads % kv != 0)
    return fail(c, JN_EINVAL, "n_kv_heads %d must divide n_heads %d", bb->n_kv_heads, bb->n_heads);
  if (bb->causal != 0 && bb->causal != 1) return fail(c, JN_EINVAL, "causal must be 0 or 1");
  if (!(bb->rope_theta >= 0.f) || std::isinf(bb->rope_theta)) return fail(c, JN_EINVAL, "rope_theta must be >= 0");
  bool glu = bb->layers[0].w_gate != nullptr;
  for (int l = 0; l < bb->n_layers; ++l) {
    const jn_layer& L = bb->layers[l];
    if (!L.wqkv || !L.wo || !L.w_up || !L.w_down || !L.g1 || !L.g2)
      return fail(c, JN_EINVAL, "layer %d has a null weight", l);
    if ((L.w_gate != nullptr) != glu) return fail(c, JN_EINVAL, "layer %d mixes GELU and GeGLU MLPs", l);
    const void* ps[] = {L.wqkv, L.wo, L.w_up, L.w_down, L.w_gate};
    for (const void* q : ps)
      if (q && ((uintptr_t)q) % 16 != 0) return fail(c, JN_EUNSUPPORTED, "layer %d weight not 16-byte aligned", l);
  }
  return JN_OK;
}

}  // namespace

jn_status jn_backbone_workspace_size(const jn_backbone* bb, int32_t T, size_t* bytes) {
  if (!bb || !bytes || T < 0) return JN_EINVAL;
  *bytes = bb_layout(bb, T).total;
  return JN_OK;
}

jn_status jn_backbone_forward(jn_ctx* c, const jn_backbone* bb, const jn_packed* p, void* hidden, void* ws,
                              size_t ws_bytes) {
  if (!c) return JN_EINVAL;
  jn_status st = check_backbone(c, bb);
  if (st != JN_OK) return st;
  if (!valid_packed(p) || !p->tokens) return fail(c, JN_EINVAL, "invalid packed batch");
  if (p->d != bb->d) return fail(c, JN_EINCOMPAT, "packed width %d != backbone width %d", p->d, bb->d);
  if (!hidden || !ws) return fail(c, JN_EINVAL, "null hidden or workspace");
  BbLayout L = bb_layout(bb, p->T);
  if (ws_bytes < L.total) return fail(c, JN_ENOSPACE, "workspace %zu B < %zu B", ws_bytes, L.total);
  if (((uintptr_t)ws) % 256 != 0 || ((uintptr_t)hidden) % 16 != 0)
    return fail(c, JN_EUNSUPPORTED, "workspace must be 256-byte and hidden 16-byte aligned");

  const int32_t T = p->T, d = bb->d, f = bb->ffn;
  {
    // launch-size limits, checked before anything is enqueued: a dispatch
    // holds at most 2^32 - 1 work-items (GEMM: <= 512 threads per 128x128-or-
    // larger tile), and the attention grid at most 2^30 workgroups
    const int64_t kv = bb->n_kv_heads ? bb->n_kv_heads : bb->n_heads;
    const int64_t nmax = std::max<int64_t>((bb->n_heads + 2 * kv) * (d / bb->n_heads),
                                           (bb->layers[0].w_gate ? 2 : 1) * (int64_t)f);
    const int64_t gemm_items = ((int64_t)T + 127) / 128 * ((nmax + 127) / 128) * 512;
    const int64_t qtiles = ((int64_t)p->max_seqlen + 127) / 128;
    const int64_t attn_blocks = ((int64_t)p->N * kv + 7) / 8 * 8 * (bb->n_heads / kv) * qtiles;
    if (gemm_items >= (1ll << 32) || attn_blocks > (1ll << 30))
      return fail(c, JN_ESHAPE, "batch of %d rows / %d samples exceeds one launch's grid", T, p->N);
  }
  char* w = (char*)ws;
  float* x = (float*)(w + L.x);
  void* h = w + L.h;
  void* qkv = w + L.qkv;
  void* att = w + L.att;
  void* mid = w + L.mid;
  void* sp = w + L.split;
  const size_t spb = L.split_bytes;
  const bool glu = bb->layers[0].w_gate != nullptr;
  const int32_t hd = d / bb->n_heads;
  const int32_t kvh = bb->n_kv_heads ? bb->n_kv_heads : bb->n_heads;
  const int32_t nqkv = (bb->n_heads + 2 * kvh) * hd;  // q | k | v columns of the projection
  hipStream_t s = c->stream;
  for (int l = 0; l < bb->n_layers; ++l) {
    const jn_layer& Ly = bb->layers[l];
    if (l == 0)
      JN_TRACED(c, JN_OP_RMSNORM, T, d, 0, launch_rmsnorm_bf16in(s, p->tokens, x, Ly.g1, h, T, d, bb->eps), "rmsnorm");
    else
      JN_TRACED(c, JN_OP_RMSNORM, T, d, 0, launch_rmsnorm_f32in(s, x, Ly.g1, h, T, d, bb->eps), "rmsnorm");
    JN_TRACED(c, JN_OP_GEMM_QKV, T, nqkv, d,
              launch_gemm(s, EPI_BF16, h, d, Ly.wqkv, nullptr, d, qkv, nqkv, T, nqkv, d, 0, sp, spb), "gemm qkv");
    if (bb->rope_theta > 0.f)
      JN_TRACED(c, JN_OP_ROPE, T, (bb->n_heads + kvh) * hd, 0,
                launch_rope(s, qkv, nqkv, p->token_pos, T, bb->n_heads + kvh, hd, bb->rope_theta), "rope");
    JN_TRACED(c, JN_OP_ATTENTION, T, d, bb->n_heads,
              launch_attention(s, qkv, att, p->seqlens, p->cu_seqlens, p->N, d, bb->n_heads, kvh, bb->causal != 0,
                               p->max_seqlen, p->align),
              "attention");
    JN_TRACED(c, JN_OP_GEMM_O, T, d, d, launch_gemm(s, EPI_RESID_F32, att, d, Ly.wo, nullptr, d, x, d, T, d, d, 0, sp, spb),
              "gemm o");
    JN_TRACED(c, JN_OP_RMSNORM, T, d, 0, launch_rmsnorm_f32in(s, x, Ly.g2, h, T, d, bb->eps), "rmsnorm");
    if (glu)
      JN_TRACED(c, JN_OP_GEMM_UP, T, 2 * f, d,
                launch_gemm(s, EPI_GEGLU_BF16, h, d, Ly.w_gate, Ly.w_up, d, mid, f, T, f, d, 0), "gemm geglu");
    else
      JN_TRACED(c, JN_OP_GEMM_UP, T, f, d, launch_gemm(s, EPI_GELU_BF16, h, d, Ly.w_up, nullptr, d, mid, f, T, f, d, 0, sp, spb),
                "gemm up");
    JN_TRACED(c, JN_OP_GEMM_DOWN, T, d, f,
              launch_gemm(s, EPI_RESID_F32, mid, f, Ly.w_down, nullptr, f, x, d, T, d, f, 0, sp, spb), "gemm down");
  }
  JN_TRACED(c, JN_OP_RMSNORM, T, d, 0, launch_rmsnorm_f32in(s, x, bb->gf, hidden, T, d, bb->eps), "final rmsnorm");
  return JN_OK;
}

// ----------------------------------------------------------------- heads ---

namespace {

struct HeadPlan {
  int maxL = 0;
  std::vector<int64_t> width;      // per layer index k: max output width
  size_t P = 0, Z0 = 0, total = 0; // offsets
  std::vector<size_t> Z, H, dZ;    // per k
  size_t descs = 0, tiles = 0, part = 0, lpart = 0;
  std::vector<HeadGemm> dv;
  std::vector<HeadTile> tv;
  std::vector<LossDesc> lv;
  size_t losses = 0;
  // launch ranges into tv
  std::vector<std::pair<int32_t, int32_t>> fwd, bwd;
};

constexpr int kHTM = 32;  // fp32 head GEMM tile: rows
constexpr int kHTN = 64;  // and columns

jn_status check_heads(jn_ctx* c, const jn_packed* p, const jn_head* heads, int32_t G) {
  if (!heads) return fail(c, JN_EINVAL, "null heads");
  if (G != p->G) return fail(c, JN_EINVAL, "G=%d but the packed batch has %d tenants", G, p->G);
  for (int32_t g = 0; g < G; ++g) {
    const jn_head& H = heads[g];
    if (H.n_layers < 1 || !H.dims || !H.W || !H.b) return fail(c, JN_EINVAL, "head %d incomplete", g);
    if (H.dims[0] != p->d) return fail(c, JN_EINCOMPAT, "head %d input %d != feature width %d", g, H.dims[0], p->d);
    for (int k = 0; k <= H.n_layers; ++k)
      if (H.dims[k] < 1) return fail(c, JN_EINVAL, "head %d dims[%d] < 1", g, k);
    if ((int64_t)H.action_dim * H.chunk != H.dims[H.n_layers])
      return fail(c, JN_EINVAL, "head %d output %d != action_dim*chunk", g, H.dims[H.n_layers]);
    for (int k = 0; k < H.n_layers; ++k)
      if (!H.W[k] || !H.b[k]) return fail(c, JN_EINVAL, "head %d layer %d null weight", g, k);
  }
  return JN_OK;
}

// Workspace layout: pooled P [N][d] | per layer k: Z_k, H_k, dZ_k [N][width_k] |
// split-K partial sums (the largest ksplit x N x width of any split launch) |
// per-tenant loss partial sums (16 G floats) |
// loss descriptors | gemm descriptors | tiles.  Tenant g's rows of every
// [N][*] buffer are its tenant-order rows [off_g, off_g + n_g).
void head_layout(const jn_packed* p, const jn_head* heads, int32_t G, HeadPlan* hp, bool with_descs) {
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align_up(o + bytes, 256);
    return at;
  };
  const int64_t N = p->N;
  hp->maxL = 0;
  for (int32_t g = 0; g < G; ++g) hp->maxL = std::max(hp->maxL, heads[g].n_layers);
  hp->width.assign(hp->maxL, 0);
  for (int32_t g = 0; g < G; ++g)
    for (int k = 0; k < heads[g].n_layers; ++k) hp->width[k] = std::max<int64_t>(hp->width[k], heads[g].dims[k + 1]);
  hp->P = take(4 * N * p->d);
  hp->Z.resize(hp->maxL);
  hp->H.resize(hp->maxL);
  hp->dZ.resize(hp->maxL);
  for (int k = 0; k < hp->maxL; ++k) {
    hp->Z[k] = take(4 * N * hp->width[k]);
    hp->H[k] = take(4 * N * hp->width[k]);
    hp->dZ[k] = take(4 * N * hp->width[k]);
  }
  if (!with_descs) {
    // descriptor counts are bounded by G * 2 * maxL; tiles computed exactly below
  }
  // tile counts: fwd M-dynamic (rows bounded by the largest tenant), bwd
  // wgrad + dgrad; a split descriptor has ksplit tiles per output tile plus
  // one reduce tile
  const int64_t tm_dyn = (tenant_rows_bound(p) + kHTM - 1) / kHTM;
  int64_t ntiles = 0, ndesc = 0, part_elems = 0;
  for (int32_t g = 0; g < G; ++g) {
    const jn_head& Hh = heads[g];
    for (int k = 0; k < Hh.n_layers; ++k) {
      int64_t in = Hh.dims[k], out = Hh.dims[k + 1];
      const int64_t sf = head_ksplit(in), sd = head_ksplit(out);
      ntiles += tm_dyn * ((out + kHTN - 1) / kHTN) * (sf + (sf > 1));           // fwd
      ntiles += ((out + kHTM - 1) / kHTM) * ((in + kHTN - 1) / kHTN);           // wgrad
      if (k > 0) ntiles += tm_dyn * ((in + kHTN - 1) / kHTN) * (sd + (sd > 1)); // dgrad
      ndesc += (k > 0) ? 3 : 2;
      if (sf > 1) part_elems = std::max(part_elems, sf * N * hp->width[k]);
      if (k > 0 && sd > 1) part_elems = std::max(part_elems, sd * N * hp->width[k - 1]);
    }
  }
  hp->part = take(4 * part_elems);
  hp->lpart = take(4 * 16 * G);
  hp->losses = take(sizeof(LossDesc) * G);
  hp->descs = take(sizeof(HeadGemm) * ndesc);
  hp->tiles = take(sizeof(HeadTile) * ntiles);
  hp->total = o;
}

}  // namespace

jn_status jn_heads_workspace_size(const jn_packed* p, const jn_head* heads, int32_t G, size_t* bytes) {
  if (!bytes || !valid_packed(p)) return JN_EINVAL;
  jn_status st = check_heads(nullptr, p, heads, G);
  if (st != JN_OK) return st;
  HeadPlan hp;
  head_layout(p, heads, G, &hp, false);
  *bytes = hp.total;
  return JN_OK;
}

}  // extern "C"

namespace {

// Body of both heads entry points; `fixed` = the allocation-free variant
// (tables staged through the context's fixed pinned buffer).
jn_status heads_run(jn_ctx* c, const jn_packed* p, const void* hidden, const jn_head* heads, const jn_head_io* io,
                    int32_t G, void* ws, size_t ws_bytes, float* pooled, bool fixed) {
  if (!valid_packed(p)) return fail(c, JN_EINVAL, "invalid packed batch");
  if (!hidden || !io || !ws) return fail(c, JN_EINVAL, "null hidden, io or workspace");
  if (((uintptr_t)hidden) % 16 != 0 || p->d % 8 != 0)
    return fail(c, JN_EUNSUPPORTED, "hidden must be 16-byte aligned and d a multiple of 8");
  if ((int64_t)p->N * ((p->d + 63) / 64) > 0x7fffffff) return fail(c, JN_ESHAPE, "too many samples for the pool grid");
  jn_status st = check_heads(c, p, heads, G);
  if (st != JN_OK) return st;
  for (int32_t g = 0; g < G; ++g) {
    const jn_head_io& I = io[g];
    if (!I.targets || !I.actions || !I.loss || !I.dW || !I.db) return fail(c, JN_EINVAL, "io %d incomplete", g);
    for (int k = 0; k < heads[g].n_layers; ++k)
      if (!I.dW[k] || !I.db[k]) return fail(c, JN_EINVAL, "io %d layer %d null gradient", g, k);
  }
  HeadPlan hp;
  head_layout(p, heads, G, &hp, true);
  if (ws_bytes < hp.total) return fail(c, JN_ENOSPACE, "workspace %zu B < %zu B", ws_bytes, hp.total);
  if (((uintptr_t)ws) % 256 != 0) return fail(c, JN_EUNSUPPORTED, "workspace must be 256-byte aligned");

  char* w = (char*)ws;
  float* P = pooled ? pooled : (float*)(w + hp.P);
  const int64_t N = p->N, d = p->d;
  const int32_t tm_dyn = (int32_t)((tenant_rows_bound(p) + kHTM - 1) / kHTM);
  auto Zk = [&](int k) { return (float*)(w + hp.Z[k]); };
  auto Hk = [&](int k) { return (float*)(w + hp.H[k]); };
  auto dZk = [&](int k) { return (float*)(w + hp.dZ[k]); };

  std::vector<HeadGemm> descs;
  std::vector<HeadTile> tiles;
  std::vector<std::pair<int32_t, int32_t>> fwd_rng, bwd_rng, fwd_red, bwd_red;
  // a descriptor whose K is long enough is split into K ranges whose sums go
  // to the partial area (plane = the [N][width] extent of its C buffer)
  float* const part = (float*)(w + hp.part);
  auto split_desc = [&](HeadGemm& D, int64_t plane) {
    D.ksplit = head_ksplit(D.K);
    if (D.ksplit > 1) {
      D.part = part;
      D.part_plane = plane;
    }
  };
  // reduce tiles of the split descriptors among tiles [t0, end): appended
  // after them, returned as a range
  auto reduce_tiles = [&](int32_t t0) {
    const int32_t t1 = (int32_t)tiles.size();
    for (int32_t t = t0; t < t1; ++t)
      if (descs[tiles[t].desc].ksplit > 1 && tiles[t].tk == 0) tiles.push_back(HeadTile{tiles[t].desc, tiles[t].tm, tiles[t].tn, 0});
    return std::make_pair(t1, (int32_t)tiles.size() - t1);
  };
  // forward, one launch per layer index
  for (int k = 0; k < hp.maxL; ++k) {
    int32_t t0 = (int32_t)tiles.size();
    for (int32_t g = 0; g < G; ++g) {
      const jn_head& Hh = heads[g];
      if (k >= Hh.n_layers) continue;
      const int64_t in = Hh.dims[k], out = Hh.dims[k + 1];
      const float* X = (k == 0) ? P : Hk(k - 1);
      const int64_t ldx = (k == 0) ? d : hp.width[k - 1];
      HeadGemm D{};
      D.A = X;
      D.sam = ldx;
      D.sak = 1;
      D.B = Hh.W[k];
      D.sbk = 1;
      D.sbn = in;
      D.C = Zk(k);
      D.ldc = hp.width[k];
      D.bias = Hh.b[k];
      D.Cact = (k + 1 < Hh.n_layers) ? Hk(k) : nullptr;
      D.bumpA = ldx;
      D.bumpB = 0;
      D.bumpC = hp.width[k];
      D.M = -1;
      D.N = (int32_t)out;
      D.K = (int32_t)in;
      D.tenant = g;
      D.tiles_n = (int32_t)((out + kHTN - 1) / kHTN);
      split_desc(D, N * hp.width[k]);
      int32_t di = (int32_t)descs.size();
      descs.push_back(D);
      for (int32_t tk = 0; tk < D.ksplit; ++tk)
        for (int32_t tm = 0; tm < tm_dyn; ++tm)
          for (int32_t tn = 0; tn < D.tiles_n; ++tn) tiles.push_back(HeadTile{di, tm, tn, tk});
    }
    fwd_rng.emplace_back(t0, (int32_t)tiles.size() - t0);
    fwd_red.push_back(reduce_tiles(t0));
  }
  // loss: y = Z_{L-1} rows, dY -> dZ_{L-1}
  std::vector<LossDesc> losses(G);
  for (int32_t g = 0; g < G; ++g) {
    const int L = heads[g].n_layers;
    losses[g] = LossDesc{Zk(L - 1), io[g].targets, dZk(L - 1), io[g].loss, io[g].actions,
                         heads[g].dims[L], hp.width[L - 1], g, 0};
  }
  // backward, one launch per step s (tenant g at layer k = L_g - 1 - s)
  for (int sidx = 0; sidx < hp.maxL; ++sidx) {
    int32_t t0 = (int32_t)tiles.size();
    for (int32_t g = 0; g < G; ++g) {
      const jn_head& Hh = heads[g];
      const int k = Hh.n_layers - 1 - sidx;
      if (k < 0) continue;
      const int64_t in = Hh.dims[k], out = Hh.dims[k + 1];
      const float* X = (k == 0) ? P : Hk(k - 1);
      const int64_t ldx = (k == 0) ? d : hp.width[k - 1];
      // wgrad: dW[out][in] = sum_rows dZ[row][o] X[row][i]; db[o] = sum_rows dZ[row][o]
      HeadGemm Wg{};
      Wg.A = dZk(k);
      Wg.sam = 1;
      Wg.sak = hp.width[k];
      Wg.B = X;
      Wg.sbk = ldx;
      Wg.sbn = 1;
      Wg.C = io[g].dW[k];
      Wg.ldc = in;
      Wg.db = io[g].db[k];
      Wg.bumpA = hp.width[k];
      Wg.bumpB = ldx;
      Wg.bumpC = 0;
      Wg.M = (int32_t)out;
      Wg.N = (int32_t)in;
      Wg.K = -1;
      Wg.tenant = g;
      Wg.tiles_n = (int32_t)((in + kHTN - 1) / kHTN);
      int32_t di = (int32_t)descs.size();
      descs.push_back(Wg);
      const int32_t tmw = (int32_t)((out + kHTM - 1) / kHTM);
      for (int32_t tm = 0; tm < tmw; ++tm)
        for (int32_t tn = 0; tn < Wg.tiles_n; ++tn) tiles.push_back(HeadTile{di, tm, tn, 0});
      if (k > 0) {
        // dgrad: dZ_{k-1}[row][i] = (sum_o dZ_k[row][o] W[o][i]) * gelu'(Z_{k-1}[row][i])
        HeadGemm Dg{};
        Dg.A = dZk(k);
        Dg.sam = hp.width[k];
        Dg.sak = 1;
        Dg.B = Hh.W[k];
        Dg.sbk = in;
        Dg.sbn = 1;
        Dg.C = dZk(k - 1);
        Dg.ldc = hp.width[k - 1];
        Dg.Zg = Zk(k - 1);
        Dg.bumpA = hp.width[k];
        Dg.bumpB = 0;
        Dg.bumpC = hp.width[k - 1];
        Dg.M = -1;
        Dg.N = (int32_t)in;
        Dg.K = (int32_t)out;
        Dg.tenant = g;
        Dg.tiles_n = (int32_t)((in + kHTN - 1) / kHTN);
        split_desc(Dg, N * hp.width[k - 1]);
        int32_t dj = (int32_t)descs.size();
        descs.push_back(Dg);
        for (int32_t tk = 0; tk < Dg.ksplit; ++tk)
          for (int32_t tm = 0; tm < tm_dyn; ++tm)
            for (int32_t tn = 0; tn < Dg.tiles_n; ++tn) tiles.push_back(HeadTile{dj, tm, tn, tk});
      }
    }
    bwd_rng.emplace_back(t0, (int32_t)tiles.size() - t0);
    bwd_red.push_back(reduce_tiles(t0));
  }

  // one upload of every table: losses | descs | tiles (contiguous in ws)
  const size_t lbytes = sizeof(LossDesc) * G, dbytes = sizeof(HeadGemm) * descs.size(),
               tbytes = sizeof(HeadTile) * tiles.size();
  if (hp.descs + dbytes > hp.tiles || hp.tiles + tbytes > hp.total)
    return fail(c, JN_ENOSPACE, "internal: head table sizing");
  std::vector<char> img(hp.total - hp.losses, 0);
  std::memcpy(img.data(), losses.data(), lbytes);
  std::memcpy(img.data() + (hp.descs - hp.losses), descs.data(), dbytes);
  std::memcpy(img.data() + (hp.tiles - hp.losses), tiles.data(), tbytes);
  st = fixed ? stage_copy_fixed(c, w + hp.losses, img.data(), hp.tiles - hp.losses + tbytes)
             : stage_copy(c, w + hp.losses, img.data(), hp.tiles - hp.losses + tbytes);
  if (st != JN_OK) return st;
  const LossDesc* dl = (const LossDesc*)(w + hp.losses);
  const HeadGemm* dd = (const HeadGemm*)(w + hp.descs);
  const HeadTile* dt = (const HeadTile*)(w + hp.tiles);
  hipStream_t s = c->stream;

  JN_TRACED(c, JN_OP_POOL, p->T, p->d, p->N,
            launch_pool(s, hidden, p->seqlens, p->cu_seqlens, p->sample_tenant_rank, p->N, p->d, P), "pool");
  for (size_t i = 0; i < fwd_rng.size(); ++i) {
    const auto r = fwd_rng[i], q = fwd_red[i];
    if (r.second)
      JN_TRACED(c, JN_OP_HEAD_FWD, r.second, 0, 0, launch_head_gemm(s, dd, dt + r.first, r.second, p->tenant_sample_off),
                "head fwd");
    if (q.second)
      JN_TRACED(c, JN_OP_HEAD_FWD, q.second, 0, 0, launch_head_reduce(s, dd, dt + q.first, q.second, p->tenant_sample_off),
                "head fwd reduce");
  }
  JN_TRACED(c, JN_OP_LOSS, G, 0, 0, launch_mse(s, dl, G, p->tenant_sample_off, (float*)(w + hp.lpart)), "loss");
  for (size_t i = 0; i < bwd_rng.size(); ++i) {
    const auto r = bwd_rng[i], q = bwd_red[i];
    if (r.second)
      JN_TRACED(c, JN_OP_HEAD_BWD, r.second, 0, 0, launch_head_gemm(s, dd, dt + r.first, r.second, p->tenant_sample_off),
                "head bwd");
    if (q.second)
      JN_TRACED(c, JN_OP_HEAD_BWD, q.second, 0, 0, launch_head_reduce(s, dd, dt + q.first, q.second, p->tenant_sample_off),
                "head bwd reduce");
  }
  return JN_OK;
}

}  // namespace

extern "C" {

jn_status jn_tenant_heads_fwd_bwd(jn_ctx* c, const jn_packed* p, const void* hidden, const jn_head* heads,
                                  const jn_head_io* io, int32_t G, void* ws, size_t ws_bytes, float* pooled) {
  if (!c) return JN_EINVAL;
  return heads_run(c, p, hidden, heads, io, G, ws, ws_bytes, pooled, false);
}

jn_status jn_tenant_heads_fwd_bwd_noalloc(jn_ctx* c, const jn_packed* p, const void* hidden, const jn_head* heads,
                                          const jn_head_io* io, int32_t G, float* pooled) {
  if (!c) return JN_EINVAL;
  if (!c->scratch) return fail(c, JN_EHIP, "the library scratch array has no device address on device %d", c->device);
  if (valid_packed(p) && heads && G == p->G && check_heads(nullptr, p, heads, G) == JN_OK) {
    HeadPlan hp;
    head_layout(p, heads, G, &hp, false);
    if (hp.total > kHeadsScratchBytes)
      return fail(c, JN_ENOSPACE, "heads need %zu B of workspace; the allocation-free call has %zu B", hp.total,
                  kHeadsScratchBytes);
  }
  return heads_run(c, p, hidden, heads, io, G, c->scratch, kHeadsScratchBytes, pooled, true);
}

// ---------------------------------------------------------------- unpack ---

jn_status jn_unpack(jn_ctx* c, const jn_packed* p, const jn_request* req, int32_t R, const void* rows,
                    size_t row_bytes, void* const* req_out) {
  if (!c) return JN_EINVAL;
  if (!valid_packed(p) || !p->token_sample) return fail(c, JN_EINVAL, "invalid packed batch");
  if (!req || !rows || !req_out) return fail(c, JN_EINVAL, "null argument");
  if (R != p->R) return fail(c, JN_EINVAL, "R=%d but the packed batch has %d requests", R, p->R);
  if (row_bytes == 0 || row_bytes % 4 != 0) return fail(c, JN_EUNSUPPORTED, "row_bytes %zu not a positive multiple of 4", row_bytes);
  if (((uintptr_t)rows) % 4 != 0) return fail(c, JN_EUNSUPPORTED, "rows not 4-byte aligned");
  std::vector<ReqEntry> rt(R);
  int64_t n = 0;
  int32_t mreq = 0;
  bool vec16 = row_bytes % 16 == 0 && ((uintptr_t)rows) % 16 == 0;
  for (int32_t r = 0; r < R; ++r) {
    if (!req_out[r]) return fail(c, JN_EINVAL, "request %d output is null", r);
    if (((uintptr_t)req_out[r]) % 4 != 0) return fail(c, JN_EUNSUPPORTED, "request %d output not 4-byte aligned", r);
    vec16 = vec16 && ((uintptr_t)req_out[r]) % 16 == 0;
    if (req[r].n_samples < 1 || req[r].max_len < 1) return fail(c, JN_ESHAPE, "request %d shape", r);
    rt[r] = ReqEntry{req[r].embeds, req_out[r], req[r].max_len, req[r].n_samples, (int32_t)n, 0};
    n += req[r].n_samples;
    mreq = std::max(mreq, req[r].max_len);
  }
  if (n != p->N) return fail(c, JN_ESHAPE, "requests hold %lld samples, packed batch %d", (long long)n, p->N);
  if (request_signature(req, R) != p->req_sig)
    return fail(c, JN_ESHAPE, "requests differ from those the batch was packed from (sample counts or max_len)");
  jn_status st = stage_copy(c, p->req_table, rt.data(), sizeof(ReqEntry) * R);
  if (st != JN_OK) return st;
  JN_TRACED(c, JN_OP_UNPACK, p->T, (int64_t)row_bytes, 0, launch_unpack(c->stream, (const ReqEntry*)p->req_table, p->sample_request, p->sample_local,
                          p->seqlens, p->cu_seqlens, p->N, mreq, rows, (int64_t)row_bytes, vec16),
         "unpack kernel");
  return JN_OK;
}

}  // extern "C"

// --------------------------------------------------------- action expert ---

namespace {

// Action vectors are padded to kAP columns (zeros) and each tenant's rows to a
// multiple of kKP for the weight-gradient contractions: the GEMM's K step.
constexpr int kAP = 64;
constexpr int kKP = 64;

// K ranges of an expert weight gradient contracted over K rows (a tenant's
// action rows or its samples' prefix rows): S = round(K / 6144) ranges, 1..8,
// of ceil(K / S) rows rounded up to 64 (the last one shorter), their fp32
// partials added in range order.  A function of K only, so a tenant's
// gradient bits do not depend on the batch it runs in.  The cross-attention
// key/value weight gradient contracts over ~12K prefix rows per tenant of the
// 16-tenant workload, 1.5 waves of 256x256 tiles unsplit.
constexpr int64_t kWgradRange = 6144;
int32_t wgrad_splits(int64_t K) {
  return (int32_t)std::min<int64_t>(8, std::max<int64_t>(1, (K + kWgradRange / 2) / kWgradRange));
}
int64_t wgrad_range_rows(int64_t K, int32_t S) { return ((K + S - 1) / S + 63) / 64 * 64; }

struct ExpShape {
  int32_t L, d, H, f, chunk, dp;
  float eps;
  int32_t dt = 0;     // flow-time feature width (0: plain regression)
  int32_t ki = kAP;   // staged input width: padded actions, then flow-time features
};

// Host view of one expert call: per-tenant rows and padded contraction sizes.
struct ExpPlan {
  ExpShape sh{};
  int32_t G = 0, N = 0;
  std::vector<int32_t> rows, roff, Ka, kaoff, Kz, kzoff;
  std::vector<int64_t> Pz, zoff;
  int64_t Na = 0, Pzt = 0, KaT = 0, KzT = 0;
};

// Workspace regions (byte offsets); per-layer saves are arrays of offsets.
struct ExpLayout {
  size_t arena = 0, arena_bytes = 0;
  size_t x, xf, yb, ub, vel, predp, dpred, dpredb, z, zoff, winp, woutp, woutpT, dx, dxb, tf, dsum, tb, dkvb, gx, part,
      TA, TB, WT, kpart, dwinp, dwoutp;
  std::vector<size_t> x1, x2, x3, h1, h2, h3, qkv, os, osb, lses, qc, kv, oc, ocb, lsec, pre, mb;
  size_t total = 0;
};

jn_status exp_plan(jn_ctx* c, const jn_packed* p, const jn_expert* ex, const jn_expert_io* io, int32_t G,
                   ExpPlan* P) {
  if (!ex || !io) return fail(c, JN_EINVAL, "null experts or io");
  if (G != p->G) return fail(c, JN_EINVAL, "G=%d but the packed batch has %d tenants", G, p->G);
  const jn_expert& e0 = ex[0];
  ExpShape sh{e0.n_layers, e0.d, e0.n_heads, e0.ffn, e0.chunk, e0.d_prefix, e0.eps};
  if (sh.L < 1 || sh.d < 1 || sh.H < 1 || sh.f < 1 || sh.chunk < 1) return fail(c, JN_EINVAL, "expert sizes must be positive");
  if (sh.chunk > 64) return fail(c, JN_EUNSUPPORTED, "chunk %d > 64", sh.chunk);
  if (sh.d % sh.H != 0 || (sh.d / sh.H != 64 && sh.d / sh.H != 128))
    return fail(c, JN_EUNSUPPORTED, "expert head dim must be 64 or 128");
  if (sh.d != 256 && sh.d != 512 && sh.d != 1024 && sh.d != 2048) return fail(c, JN_EUNSUPPORTED, "expert width %d", sh.d);
  if (sh.f % 64 != 0 || sh.dp % 64 != 0) return fail(c, JN_EUNSUPPORTED, "ffn and d_prefix must be multiples of 64");
  if (sh.dp != p->d) return fail(c, JN_EINCOMPAT, "expert reads width %d, backbone has %d", sh.dp, p->d);
  if (!(sh.eps > 0.f)) return fail(c, JN_EINVAL, "eps must be > 0");
  if (e0.w_time) {
    if (e0.d_time < 64 || e0.d_time % 64 != 0 || e0.d_time > 4096)
      return fail(c, JN_EUNSUPPORTED, "d_time %d must be a multiple of 64 in [64, 4096]", e0.d_time);
    sh.dt = e0.d_time;
    sh.ki = kAP + e0.d_time;
  }
  P->sh = sh;
  P->G = G;
  P->N = p->N;
  int64_t n = 0;
  for (int32_t g = 0; g < G; ++g) {
    const jn_expert& e = ex[g];
    if (e.n_layers != sh.L || e.d != sh.d || e.n_heads != sh.H || e.ffn != sh.f || e.chunk != sh.chunk ||
        e.d_prefix != sh.dp || e.eps != sh.eps)
      return fail(c, JN_EUNSUPPORTED, "expert %d differs in shape from expert 0", g);
    if (e.action_dim < 1 || e.action_dim > 32) return fail(c, JN_EUNSUPPORTED, "expert %d action_dim %d", g, e.action_dim);
    if (!e.w_in || !e.w_out || !e.gf || !e.layers) return fail(c, JN_EINVAL, "expert %d incomplete", g);
    for (int l = 0; l < sh.L; ++l) {
      const jn_expert_layer& L = e.layers[l];
      const void* ps[] = {L.wqkv_s, L.wo_s, L.wq_c, L.wkv_c, L.wo_c, L.w_up, L.w_down, L.g1, L.g2, L.g3};
      for (const void* q : ps)
        if (!q) return fail(c, JN_EINVAL, "expert %d layer %d has a null weight", g, l);
    }
    const jn_expert_io& I = io[g];
    if (I.n_samples < 1 || I.prefix_rows < I.n_samples) return fail(c, JN_ESHAPE, "io %d sizes", g);
    if (!I.noisy || !I.targets || !I.pred || !I.loss || !I.dw_in || !I.dw_out || !I.dgf || !I.layers)
      return fail(c, JN_EINVAL, "io %d incomplete", g);
    if ((e.w_time != nullptr) != (sh.dt > 0) || (sh.dt > 0 && e.d_time != sh.dt))
      return fail(c, JN_EUNSUPPORTED, "expert %d differs from expert 0 in its flow-time projection", g);
    if (sh.dt > 0 && (!I.flow_t || !I.dw_time || ((uintptr_t)I.dw_time) % 16 != 0))
      return fail(c, JN_EINVAL, "io %d: flow matching needs flow_t and an aligned dw_time", g);
    if (sh.dt == 0 && (I.flow_t || I.dw_time))
      return fail(c, JN_EINVAL, "io %d: flow_t / dw_time given but expert %d has no w_time", g, g);
    for (int l = 0; l < sh.L; ++l) {
      const jn_expert_layer_grads& Gr = I.layers[l];
      float* ps[] = {Gr.wqkv_s, Gr.wo_s, Gr.wq_c, Gr.wkv_c, Gr.wo_c, Gr.w_up, Gr.w_down, Gr.g1, Gr.g2, Gr.g3};
      for (float* q : ps)
        if (!q || ((uintptr_t)q) % 16 != 0) return fail(c, JN_EINVAL, "io %d layer %d gradient null or unaligned", g, l);
    }
    n += I.n_samples;
  }
  if (n != p->N) return fail(c, JN_ESHAPE, "io holds %lld samples, packed batch %d", (long long)n, p->N);
  P->rows.resize(G);
  P->roff.assign(G + 1, 0);
  P->Ka.resize(G);
  P->kaoff.assign(G + 1, 0);
  P->Kz.resize(G);
  P->kzoff.assign(G + 1, 0);
  P->Pz.resize(G);
  P->zoff.assign(G + 1, 0);
  for (int32_t g = 0; g < G; ++g) {
    P->rows[g] = io[g].n_samples * sh.chunk;
    P->roff[g + 1] = P->roff[g] + P->rows[g];
    P->Ka[g] = (P->rows[g] + kKP - 1) / kKP * kKP;
    P->kaoff[g + 1] = P->kaoff[g] + P->Ka[g];
    P->Pz[g] = io[g].prefix_rows;
    P->zoff[g + 1] = P->zoff[g] + P->Pz[g];
    P->Kz[g] = (int32_t)((P->Pz[g] + kKP - 1) / kKP * kKP);
    P->kzoff[g + 1] = P->kzoff[g] + P->Kz[g];
  }
  P->Na = P->roff[G];
  P->Pzt = P->zoff[G];
  P->KaT = P->kaoff[G];
  P->KzT = P->kzoff[G];
  if (P->Pzt > p->T) return fail(c, JN_ESHAPE, "io prefix rows exceed the packed batch");
  if (P->Na >= (1ll << 31) || P->Pzt * 2 * sh.d >= (1ll << 40)) return fail(c, JN_ESHAPE, "expert batch too large");
  return JN_OK;
}

ExpLayout exp_layout(const ExpPlan& P) {
  ExpLayout Ly;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align_up(o + bytes, 256);
    return at;
  };
  const ExpShape& s = P.sh;
  const int64_t Na = P.Na, Pz = P.Pzt, d = s.d, f = s.f, H = s.H, G = P.G;
  const int64_t wmax = std::max<int64_t>(3 * d, f);
  Ly.arena_bytes = (size_t)(64 * s.L + 64) * G * 224 + (1 << 16);
  Ly.arena = take(Ly.arena_bytes);
  Ly.x = take(4 * Na * d);
  Ly.xf = take(4 * Na * d);
  Ly.yb = take(2 * Na * d);
  const int64_t KI = s.ki;
  Ly.ub = take(2 * Na * KI);
  Ly.vel = take(s.dt > 0 ? 4 * Na * 32 : 0);
  Ly.predp = take(4 * Na * kAP);
  Ly.dpred = take(4 * Na * kAP);
  Ly.dpredb = take(2 * Na * kAP);
  Ly.z = take(2 * Pz * s.dp);
  Ly.zoff = take(4 * (P.N + 1));
  Ly.winp = take(2 * G * d * KI);
  Ly.woutp = take(2 * G * kAP * d);
  Ly.woutpT = take(2 * G * d * kAP);
  Ly.dx = take(4 * Na * d);
  Ly.dxb = take(2 * Na * d);
  Ly.tf = take(4 * Na * d);
  Ly.dsum = take(4 * Na * H);
  Ly.tb = take(2 * Na * wmax);
  Ly.dkvb = take(2 * Pz * 2 * d);
  Ly.gx = take(4 * Na * d);
  Ly.part = take(4 * G * 16 * d);
  Ly.TA = take(2 * std::max<int64_t>(wmax * P.KaT, 2 * d * P.KzT));
  Ly.TB = take(2 * std::max<int64_t>(std::max<int64_t>(wmax, KI) * P.KaT, (int64_t)s.dp * P.KzT));
  Ly.WT = take(2 * G * std::max<int64_t>(f * d, 3 * d * d) + 2 * G * 2 * d * s.dp);
  {
    // partials of split weight gradients: action-row ones (any weight shape)
    // and prefix-row ones (the key/value weights), never live together
    const int64_t apair = std::max<int64_t>(std::max<int64_t>(f * d, 3 * d * d), std::max<int64_t>(d * KI, kAP * d));
    int64_t ka = 0, kz = 0;
    for (int32_t g = 0; g < G; ++g) {
      const int32_t Sa = wgrad_splits(P.rows[g]), Sz = wgrad_splits(P.Pz[g]);
      if (Sa > 1) ka += Sa * apair;
      if (Sz > 1) kz += Sz * 2 * d * s.dp;
    }
    Ly.kpart = take(4 * std::max(ka, kz));
  }
  Ly.dwinp = take(4 * G * d * KI);
  Ly.dwoutp = take(4 * G * kAP * d);
  for (int l = 0; l < s.L; ++l) {
    Ly.x1.push_back(take(4 * Na * d));
    Ly.x2.push_back(take(4 * Na * d));
    Ly.x3.push_back(take(4 * Na * d));
    Ly.h1.push_back(take(2 * Na * d));
    Ly.h2.push_back(take(2 * Na * d));
    Ly.h3.push_back(take(2 * Na * d));
    Ly.qkv.push_back(take(2 * Na * 3 * d));
    Ly.os.push_back(take(4 * Na * d));
    Ly.osb.push_back(take(2 * Na * d));
    Ly.lses.push_back(take(4 * Na * H));
    Ly.qc.push_back(take(2 * Na * d));
    Ly.kv.push_back(take(2 * Pz * 2 * d));
    Ly.oc.push_back(take(4 * Na * d));
    Ly.ocb.push_back(take(2 * Na * d));
    Ly.lsec.push_back(take(4 * Na * H));
    Ly.pre.push_back(take(4 * Na * f));
    Ly.mb.push_back(take(2 * Na * f));
  }
  Ly.total = o;
  return Ly;
}

// Records grouped launches: descriptor tables go to a host image of the arena,
// the launches run after one upload of that image.
struct Recorder {
  std::vector<char> img;
  size_t cap = 0;
  bool overflow = false;
  bool bad_gemm = false;
  std::vector<std::function<hipError_t(char*)>> ops;
  std::vector<int32_t> opcode;
  size_t add(const void* src, size_t bytes) {
    size_t at = align_up(img.size(), 256);
    if (at + bytes > cap) {
      overflow = true;
      return 0;
    }
    img.resize(at + bytes);
    std::memcpy(img.data() + at, src, bytes);
    return at;
  }
};

}  // namespace

extern "C" {

jn_status jn_pack_tenant_sizes(const jn_request* req, int32_t R, const jn_tenant* ten, int32_t G,
                               const jn_pack_opts* o, int32_t* samples, int64_t* rows) {
  if (!samples || !rows) return JN_EINVAL;
  Plan p;
  jn_status st = make_plan(nullptr, req, R, ten, G, o, &p);
  if (st != JN_OK) return st;
  for (int32_t g = 0; g < G; ++g) {
    samples[g] = 0;
    rows[g] = 0;
  }
  for (int32_t i = 0; i < p.N; ++i) {
    samples[p.sten[i]] += 1;
    rows[p.sten[i]] += p.seqlens[i];
  }
  return JN_OK;
}

jn_status jn_experts_workspace_size(const jn_packed* p, const jn_expert* ex, const jn_expert_io* io, int32_t G,
                                    size_t* bytes) {
  if (!bytes || !valid_packed(p)) return JN_EINVAL;
  ExpPlan P;
  jn_status st = exp_plan(nullptr, p, ex, io, G, &P);
  if (st != JN_OK) return st;
  *bytes = exp_layout(P).total;
  return JN_OK;
}

jn_status jn_tenant_experts_fwd_bwd(jn_ctx* c, const jn_packed* p, const void* hidden, const jn_expert* ex,
                                    const jn_expert_io* io, int32_t G, void* ws, size_t ws_bytes) {
  if (!c) return JN_EINVAL;
  if (!valid_packed(p) || !p->tenant_perm) return fail(c, JN_EINVAL, "invalid packed batch");
  if (!hidden || !ws) return fail(c, JN_EINVAL, "null hidden or workspace");
  ExpPlan P;
  jn_status st = exp_plan(c, p, ex, io, G, &P);
  if (st != JN_OK) return st;
  const ExpLayout Ly = exp_layout(P);
  if (ws_bytes < Ly.total) return fail(c, JN_ENOSPACE, "workspace %zu B < %zu B", ws_bytes, Ly.total);
  if (((uintptr_t)ws) % 256 != 0) return fail(c, JN_EUNSUPPORTED, "workspace must be 256-byte aligned");

  char* w = (char*)ws;
  char* const darena = w + Ly.arena;
  const ExpShape& S = P.sh;
  const int64_t d = S.d, f = S.f, dp = S.dp, H = S.H;
  const bool flow = S.dt > 0;
  const int64_t KI = S.ki;  // staged input width
  auto F = [&](size_t off) { return (float*)(w + off); };
  auto B = [&](size_t off) { return (uint16_t*)(w + off); };
  Recorder rec;
  rec.cap = Ly.arena_bytes;
  const size_t roff_at = rec.add(P.roff.data(), 4 * P.roff.size());
  hipStream_t s = c->stream;

  // ---- recording helpers
  auto gemm = [&](int epi, std::vector<GemmArgs> probs) {
    const int shape = gemm_grouped_tile_shape(probs.data(), (int32_t)probs.size());
    const int32_t tiles = gemm_grouped_prepare(probs.data(), (int32_t)probs.size(), shape);
    if (tiles < 0) rec.bad_gemm = true;
    const size_t at = rec.add(probs.data(), sizeof(GemmArgs) * probs.size());
    const int32_t n = (int32_t)probs.size();
    const int trans = probs.empty() ? 0 : probs[0].trans;
    rec.ops.push_back(
        [=](char* a) { return launch_gemm_grouped(s, epi, (const GemmArgs*)(a + at), n, tiles, shape, trans); });
    rec.opcode.push_back(JN_OP_EXPERT_GEMM);
  };
  // Transposed-operand problems run only on the 256x256 tiles; elsewhere
  // (offsets beyond the loop's 32-bit ones) the caller materialises the
  // transposes instead.  Both give the same MFMA sequence per output element.
  auto trans_ok = [&](const std::vector<GemmArgs>& probs) {
    return !c->expert_transposes && gemm_grouped_tile_shape(probs.data(), (int32_t)probs.size()) == 0;
  };
  auto per_tenant_gemm = [&](int epi, std::function<GemmArgs(int32_t)> fn) {
    std::vector<GemmArgs> v;
    for (int32_t g = 0; g < G; ++g) v.push_back(fn(g));
    gemm(epi, v);
  };
  auto copy = [&](std::vector<CopyDesc> dv) {
    const int32_t blocks = copy2d_prepare(dv.data(), (int32_t)dv.size());
    const size_t at = rec.add(dv.data(), sizeof(CopyDesc) * dv.size());
    const int32_t n = (int32_t)dv.size();
    rec.ops.push_back([=](char* a) { return launch_copy2d(s, (const CopyDesc*)(a + at), n, blocks); });
    rec.opcode.push_back(JN_OP_EXPERT_OTHER);
  };
  auto trans = [&](std::vector<TransDesc> dv) {
    const int32_t blocks = transpose_prepare(dv.data(), (int32_t)dv.size());
    const size_t at = rec.add(dv.data(), sizeof(TransDesc) * dv.size());
    const int32_t n = (int32_t)dv.size();
    rec.ops.push_back([=](char* a) { return launch_transpose(s, (const TransDesc*)(a + at), n, blocks); });
    rec.opcode.push_back(JN_OP_EXPERT_OTHER);
  };
  auto ksum = [&](std::vector<KSumDesc> dv) {
    const int32_t blocks = ksum_prepare(dv.data(), (int32_t)dv.size());
    if (blocks < 0) rec.bad_gemm = true;
    const size_t at = rec.add(dv.data(), sizeof(KSumDesc) * dv.size());
    const int32_t n = (int32_t)dv.size();
    rec.ops.push_back([=](char* a) { return launch_ksum(s, (const KSumDesc*)(a + at), n, blocks); });
    rec.opcode.push_back(JN_OP_EXPERT_OTHER);
  };
  auto ptr_table = [&](std::function<const void*(int32_t)> fn) {
    std::vector<const void*> v(G);
    for (int32_t g = 0; g < G; ++g) v[g] = fn(g);
    return rec.add(v.data(), sizeof(void*) * G);
  };
  auto rms_fwd = [&](size_t x_at, size_t gains_at, size_t h_at) {
    const int64_t rows = P.Na;
    rec.ops.push_back([=](char* a) {
      return launch_xrms_fwd(s, F(x_at), (const void* const*)(a + gains_at), (const int32_t*)(a + roff_at), G,
                             (int32_t)rows, (int32_t)d, S.eps, w + h_at);
    });
    rec.opcode.push_back(JN_OP_EXPERT_OTHER);
  };
  auto rms_bwd = [&](size_t x_at, size_t gains_at, size_t dg_at) {
    const int64_t rows = P.Na;
    rec.ops.push_back([=](char* a) {
      return launch_xrms_bwd(s, F(x_at), (const void* const*)(a + gains_at), (const int32_t*)(a + roff_at), G,
                             (int32_t)rows, (int32_t)d, S.eps, F(Ly.tf), F(Ly.dx), F(Ly.gx), F(Ly.part),
                             (float* const*)(a + dg_at));
    });
    rec.opcode.push_back(JN_OP_EXPERT_OTHER);
  };
  auto attn = [&](AttnArgs A, bool bwd) {
    const int32_t n = P.N;
    rec.ops.push_back([=](char*) { return launch_xattn(s, A, n, bwd); });
    rec.opcode.push_back(JN_OP_EXPERT_ATTENTION);
  };
  // whole-buffer copy / conversion of Na rows
  auto rows_copy = [&](const void* src, bool sb, void* dst, bool db, int64_t rows, int64_t cols) {
    CopyDesc cd{};
    cd.src = src;
    cd.dst = dst;
    cd.src_ld = cols;
    cd.dst_ld = cols;
    cd.rows = (int32_t)rows;
    cd.cols = (int32_t)cols;
    cd.src_rows = src ? (int32_t)rows : 0;
    cd.src_cols = (int32_t)cols;
    cd.src_bf16 = sb;
    cd.dst_bf16 = db;
    copy({cd});
  };
  // transpose a [rows_g][width] per-tenant block of a row buffer (ld = width)
  // into `dst_at` as [width][K_g] blocks (K padded with zeros)
  auto trans_rows = [&](const uint16_t* src, int64_t width, uint16_t* dst, bool prefix) {
    std::vector<TransDesc> v;
    for (int32_t g = 0; g < G; ++g) {
      TransDesc t{};
      const int64_t r0 = prefix ? P.zoff[g] : P.roff[g];
      const int64_t k0 = prefix ? P.kzoff[g] : P.kaoff[g];
      t.src = src + r0 * width;
      t.src_ld = width;
      t.rows = prefix ? (int32_t)P.Pz[g] : P.rows[g];
      t.cols = (int32_t)width;
      t.rows_pad = prefix ? P.Kz[g] : P.Ka[g];
      t.dst = dst + width * k0;
      t.dst_ld = t.rows_pad;
      v.push_back(t);
    }
    trans(v);
  };
  // transposed copy of each tenant's weight [rows][cols] -> WT block [cols][rows]
  auto trans_w = [&](std::function<const void*(int32_t)> wsel, int64_t rows, int64_t cols) {
    std::vector<TransDesc> v;
    for (int32_t g = 0; g < G; ++g) {
      TransDesc t{};
      t.src = (const uint16_t*)wsel(g);
      t.src_ld = cols;
      t.rows = (int32_t)rows;
      t.cols = (int32_t)cols;
      t.rows_pad = (int32_t)rows;
      t.dst = B(Ly.WT) + (int64_t)g * rows * cols;
      t.dst_ld = rows;
      v.push_back(t);
    }
    trans(v);
  };
  auto WTg = [&](int32_t g, int64_t rows, int64_t cols) { return B(Ly.WT) + (int64_t)g * rows * cols; };
  // data GEMM over each tenant's rows: C[rows][N] = X[rows][K] W[N][K]^T
  auto rows_gemm = [&](int epi, const uint16_t* X, int64_t K, std::function<const uint16_t*(int32_t)> Wsel, int64_t N,
                       void* C, int64_t ldc, bool cfp32, float* aux = nullptr) {
    per_tenant_gemm(epi, [&](int32_t g) {
      GemmArgs a{};
      a.X = X + (int64_t)P.roff[g] * K;
      a.ldx = K;
      a.W = Wsel(g);
      a.ldw = K;
      a.C = cfp32 ? (void*)((float*)C + (int64_t)P.roff[g] * ldc) : (void*)((uint16_t*)C + (int64_t)P.roff[g] * ldc);
      a.ldc = ldc;
      if (aux) {
        a.aux = aux + (int64_t)P.roff[g] * N;
        a.ldaux = N;
      }
      a.M = P.rows[g];
      a.N = (int32_t)N;
      a.K = (int32_t)K;
      return a;
    });
  };
  // weight gradient C_g[out][in] = dY_g^T X_g over the tenant's rows of two
  // row buffers (dY [rows][out], X [rows][in]; prefix: the tenant's prefix
  // rows), read transposed by the GEMM -- or from zero-padded transposes
  // (TA_g [out][K_g], TB_g [in][K_g]) -- in the K ranges of wgrad_splits
  auto wgrad_rows = [&](const uint16_t* dy, int64_t out, const uint16_t* xin, int64_t in,
                        std::function<float*(int32_t)> Csel, bool prefix) {
    std::vector<GemmArgs> vt, vm;  // transposed loads / materialised transposes
    std::vector<KSumDesc> sums;
    int64_t planes = 0;  // partial planes handed out
    for (int32_t g = 0; g < G; ++g) {
      const int64_t K = prefix ? P.Pz[g] : P.rows[g];
      const int64_t r0 = prefix ? P.zoff[g] : P.roff[g];
      const int64_t kz0 = prefix ? P.kzoff[g] : P.kaoff[g];
      const int64_t Kp = prefix ? P.Kz[g] : P.Ka[g];
      const int32_t S = wgrad_splits(K);
      const int64_t len = S > 1 ? wgrad_range_rows(K, S) : K;
      float* part = F(Ly.kpart) + planes * out * in;
      for (int32_t r = 0; r < S; ++r) {
        const int64_t k0 = r * len, k1 = r == S - 1 ? K : (r + 1) * len;
        GemmArgs a{};
        a.C = S > 1 ? (void*)(part + r * out * in) : (void*)Csel(g);
        a.ldc = in;
        a.M = (int32_t)out;
        a.N = (int32_t)in;
        a.X = dy + (r0 + k0) * out;
        a.ldx = out;
        a.W = xin + (r0 + k0) * in;
        a.ldw = in;
        a.K = (int32_t)(k1 - k0);
        a.trans = GEMM_TRANS_X | GEMM_TRANS_W;
        vt.push_back(a);
        GemmArgs m = a;  // columns k0.. of the tenant's [out][Kp] / [in][Kp] transposed blocks
        m.trans = 0;
        m.X = B(Ly.TA) + out * kz0 + k0;
        m.ldx = Kp;
        m.W = B(Ly.TB) + in * kz0 + k0;
        m.ldw = Kp;
        m.K = (int32_t)((r == S - 1 ? Kp : k1) - k0);
        vm.push_back(m);
      }
      if (S > 1) {
        sums.push_back(KSumDesc{part, Csel(g), out * in, S, 0});
        planes += S;
      }
    }
    if (trans_ok(vt)) {
      gemm(EPI_F32, vt);
    } else {
      trans_rows(dy, out, B(Ly.TA), prefix);
      trans_rows(xin, in, B(Ly.TB), prefix);
      gemm(EPI_F32, vm);
    }
    if (!sums.empty()) ksum(sums);
  };
  // data gradient C[rows][in] = epi(dY[rows][out] W_g[out][in]) per tenant,
  // the weight read transposed by the GEMM -- or from a transposed copy
  auto dgrad_rows = [&](int epi, const uint16_t* dy, int64_t out, std::function<const void*(int32_t)> wsel, int64_t in,
                        void* C, bool cfp32, float* aux = nullptr) {
    std::vector<GemmArgs> v;
    for (int32_t g = 0; g < G; ++g) {
      GemmArgs a{};
      a.X = dy + (int64_t)P.roff[g] * out;
      a.ldx = out;
      a.W = (const uint16_t*)wsel(g);
      a.ldw = in;
      a.C = cfp32 ? (void*)((float*)C + (int64_t)P.roff[g] * in) : (void*)((uint16_t*)C + (int64_t)P.roff[g] * in);
      a.ldc = in;
      if (aux) {
        a.aux = aux + (int64_t)P.roff[g] * in;
        a.ldaux = in;
      }
      a.M = P.rows[g];
      a.N = (int32_t)in;
      a.K = (int32_t)out;
      a.trans = GEMM_TRANS_W;
      v.push_back(a);
    }
    if (trans_ok(v)) {
      gemm(epi, v);
      return;
    }
    trans_w(wsel, out, in);
    rows_gemm(epi, dy, out, [&](int32_t g) { return (const uint16_t*)WTg(g, out, in); }, in, C, in, cfp32, aux);
  };
  auto Wl = [&](int l, const void* jn_expert_layer::*m) {
    return [=](int32_t g) { return (const uint16_t*)(ex[g].layers[l].*m); };
  };
  auto Gl = [&](int l, float* jn_expert_layer_grads::*m) { return [=](int32_t g) { return io[g].layers[l].*m; }; };

  // ---------------------------------------------------------------- forward
  {
    std::vector<CopyDesc> v;
    for (int32_t g = 0; g < G; ++g) {
      const int32_t a = ex[g].action_dim;
      if (!flow) {
        CopyDesc u{io[g].noisy, B(Ly.ub) + (int64_t)P.roff[g] * KI, a, KI, P.rows[g], kAP, P.rows[g], a, 0, 1, 0, 0};
        v.push_back(u);
      }
      CopyDesc wi{ex[g].w_in, B(Ly.winp) + (int64_t)g * d * KI, a, KI, (int32_t)d, kAP, (int32_t)d, a, 1, 1, 0, 0};
      CopyDesc wo{ex[g].w_out, B(Ly.woutp) + (int64_t)g * kAP * d, d, d, kAP, (int32_t)d, a, (int32_t)d, 1, 1, 0, 0};
      v.push_back(wi);
      v.push_back(wo);
      if (flow)  // the flow-time projection occupies input columns kAP .. kAP + d_time
        v.push_back(CopyDesc{ex[g].w_time, B(Ly.winp) + (int64_t)g * d * KI + kAP, S.dt, KI, (int32_t)d, S.dt,
                             (int32_t)d, S.dt, 1, 1, 0, 0});
    }
    copy(v);
    if (flow) {
      std::vector<FlowDesc> fv(G);
      for (int32_t g = 0; g < G; ++g)
        fv[g] = FlowDesc{io[g].flow_t, io[g].noisy, io[g].targets, F(Ly.vel) + (int64_t)P.roff[g] * 32,
                         (int64_t)P.roff[g], P.rows[g], ex[g].action_dim};
      const size_t at = rec.add(fv.data(), sizeof(FlowDesc) * G);
      const int64_t na = P.Na;
      const int32_t ch = S.chunk, dt = S.dt;
      uint16_t* const ubp = B(Ly.ub);
      rec.ops.push_back([=](char* ar) {
        return launch_flow_prep(s, (const FlowDesc*)(ar + at), G, na, ch, kAP, dt, ubp, (int32_t)KI);
      });
      rec.opcode.push_back(JN_OP_EXPERT_OTHER);
    }
    std::vector<TransDesc> t;
    for (int32_t g = 0; g < G; ++g)
      t.push_back(TransDesc{B(Ly.woutp) + (int64_t)g * kAP * d, B(Ly.woutpT) + (int64_t)g * d * kAP, d, kAP, kAP,
                            (int32_t)d, kAP, 0});
    trans(t);
    const int64_t cap = P.Pzt;
    rec.ops.push_back([=](char*) {
      return launch_prefix(s, hidden, p->tenant_perm, p->seqlens, p->cu_seqlens, p->N, p->max_seqlen, (int32_t)dp, cap,
                           (int32_t*)(w + Ly.zoff), w + Ly.z);
    });
    rec.opcode.push_back(JN_OP_EXPERT_OTHER);
    rows_gemm(EPI_F32, B(Ly.ub), KI, [&](int32_t g) { return B(Ly.winp) + (int64_t)g * d * KI; }, d, F(Ly.x), d, true);
  }
  const float scale = 1.0f / sqrtf((float)(d / H));
  for (int l = 0; l < S.L; ++l) {
    const size_t g1 = ptr_table([&](int32_t g) { return ex[g].layers[l].g1; });
    const size_t g2 = ptr_table([&](int32_t g) { return ex[g].layers[l].g2; });
    const size_t g3 = ptr_table([&](int32_t g) { return ex[g].layers[l].g3; });
    // self-attention block
    rows_copy(F(Ly.x), false, F(Ly.x1[l]), false, P.Na, d);
    rms_fwd(Ly.x1[l], g1, Ly.h1[l]);
    rows_gemm(EPI_BF16, B(Ly.h1[l]), d, Wl(l, &jn_expert_layer::wqkv_s), 3 * d, B(Ly.qkv[l]), 3 * d, false);
    {
      AttnArgs A{};
      A.Q = B(Ly.qkv[l]);
      A.K = B(Ly.qkv[l]);
      A.V = B(Ly.qkv[l]);
      A.O = F(Ly.os[l]);
      A.Ob = B(Ly.osb[l]);
      A.lse = F(Ly.lses[l]);
      A.ldq = 3 * d;
      A.ldkv = 3 * d;
      A.ldo = d;
      A.kcol = (int32_t)d;
      A.vcol = (int32_t)(2 * d);
      A.Lq = S.chunk;
      A.max_lk = S.chunk;
      A.hd = (int32_t)(d / H);
      A.nheads = (int32_t)H;
      A.scale = scale;
      attn(A, false);
    }
    rows_gemm(EPI_RESID_F32, B(Ly.osb[l]), d, Wl(l, &jn_expert_layer::wo_s), d, F(Ly.x), d, true);
    // cross-attention block
    rows_copy(F(Ly.x), false, F(Ly.x2[l]), false, P.Na, d);
    rms_fwd(Ly.x2[l], g2, Ly.h2[l]);
    rows_gemm(EPI_BF16, B(Ly.h2[l]), d, Wl(l, &jn_expert_layer::wq_c), d, B(Ly.qc[l]), d, false);
    per_tenant_gemm(EPI_BF16, [&](int32_t g) {
      GemmArgs a{};
      a.X = B(Ly.z) + P.zoff[g] * dp;
      a.ldx = dp;
      a.W = (const uint16_t*)ex[g].layers[l].wkv_c;
      a.ldw = dp;
      a.C = B(Ly.kv[l]) + P.zoff[g] * 2 * d;
      a.ldc = 2 * d;
      a.M = (int32_t)P.Pz[g];
      a.N = (int32_t)(2 * d);
      a.K = (int32_t)dp;
      return a;
    });
    {
      AttnArgs A{};
      A.Q = B(Ly.qc[l]);
      A.K = B(Ly.kv[l]);
      A.V = B(Ly.kv[l]);
      A.O = F(Ly.oc[l]);
      A.Ob = B(Ly.ocb[l]);
      A.lse = F(Ly.lsec[l]);
      A.zoff = (const int32_t*)(w + Ly.zoff);
      A.kv_cap = P.Pzt;
      A.ldq = d;
      A.ldkv = 2 * d;
      A.ldo = d;
      A.kcol = 0;
      A.vcol = (int32_t)d;
      A.Lq = S.chunk;
      A.max_lk = p->max_seqlen;
      A.hd = (int32_t)(d / H);
      A.nheads = (int32_t)H;
      A.scale = scale;
      attn(A, false);
    }
    rows_gemm(EPI_RESID_F32, B(Ly.ocb[l]), d, Wl(l, &jn_expert_layer::wo_c), d, F(Ly.x), d, true);
    // MLP block
    rows_copy(F(Ly.x), false, F(Ly.x3[l]), false, P.Na, d);
    rms_fwd(Ly.x3[l], g3, Ly.h3[l]);
    rows_gemm(EPI_GELU_SAVE, B(Ly.h3[l]), d, Wl(l, &jn_expert_layer::w_up), f, B(Ly.mb[l]), f, false, F(Ly.pre[l]));
    rows_gemm(EPI_RESID_F32, B(Ly.mb[l]), f, Wl(l, &jn_expert_layer::w_down), d, F(Ly.x), d, true);
  }
  const size_t gfa = ptr_table([&](int32_t g) { return ex[g].gf; });
  rows_copy(F(Ly.x), false, F(Ly.xf), false, P.Na, d);
  rms_fwd(Ly.xf, gfa, Ly.yb);
  rows_gemm(EPI_F32, B(Ly.yb), d, [&](int32_t g) { return B(Ly.woutp) + (int64_t)g * kAP * d; }, kAP, F(Ly.predp),
            kAP, true);
  {
    std::vector<XLossDesc> v(G);
    for (int32_t g = 0; g < G; ++g)
      v[g] = XLossDesc{flow ? F(Ly.vel) + (int64_t)P.roff[g] * 32 : io[g].targets, io[g].pred, io[g].loss,
                       ex[g].action_dim, 0};
    const size_t at = rec.add(v.data(), sizeof(XLossDesc) * G);
    rec.ops.push_back([=](char* a) {
      return launch_xloss(s, (const XLossDesc*)(a + at), (const int32_t*)(a + roff_at), G, F(Ly.predp), kAP,
                          F(Ly.dpred));
    });
    rec.opcode.push_back(JN_OP_LOSS);
  }

  // --------------------------------------------------------------- backward
  rows_copy(F(Ly.dpred), false, B(Ly.dpredb), true, P.Na, kAP);
  wgrad_rows(B(Ly.dpredb), kAP, B(Ly.yb), d, [&](int32_t g) { return F(Ly.dwoutp) + (int64_t)g * kAP * d; }, false);
  rows_gemm(EPI_F32, B(Ly.dpredb), kAP, [&](int32_t g) { return B(Ly.woutpT) + (int64_t)g * d * kAP; }, d, F(Ly.tf),
            d, true);
  rows_copy(nullptr, false, F(Ly.dx), false, P.Na, d);  // dx = 0
  rms_bwd(Ly.xf, gfa, ptr_table([&](int32_t g) { return (const void*)io[g].dgf; }));
  for (int l = S.L - 1; l >= 0; --l) {
    const size_t g1 = ptr_table([&](int32_t g) { return ex[g].layers[l].g1; });
    const size_t g2 = ptr_table([&](int32_t g) { return ex[g].layers[l].g2; });
    const size_t g3 = ptr_table([&](int32_t g) { return ex[g].layers[l].g3; });
    // MLP block: x += m W_down^T, m = gelu(h3 W_up^T)
    rows_copy(F(Ly.dx), false, B(Ly.dxb), true, P.Na, d);
    wgrad_rows(B(Ly.dxb), d, B(Ly.mb[l]), f, Gl(l, &jn_expert_layer_grads::w_down), false);
    dgrad_rows(EPI_GELUGRAD_BF16, B(Ly.dxb), d, [&](int32_t g) { return ex[g].layers[l].w_down; }, f, B(Ly.tb), false,
               F(Ly.pre[l]));
    wgrad_rows(B(Ly.tb), f, B(Ly.h3[l]), d, Gl(l, &jn_expert_layer_grads::w_up), false);
    dgrad_rows(EPI_F32, B(Ly.tb), f, [&](int32_t g) { return ex[g].layers[l].w_up; }, d, F(Ly.tf), true);
    rms_bwd(Ly.x3[l], g3, ptr_table([&](int32_t g) { return (const void*)io[g].layers[l].g3; }));
    // cross-attention block
    rows_copy(F(Ly.dx), false, B(Ly.dxb), true, P.Na, d);
    wgrad_rows(B(Ly.dxb), d, B(Ly.ocb[l]), d, Gl(l, &jn_expert_layer_grads::wo_c), false);
    dgrad_rows(EPI_F32, B(Ly.dxb), d, [&](int32_t g) { return ex[g].layers[l].wo_c; }, d, F(Ly.tf), true);
    {
      AttnArgs A{};
      A.Q = B(Ly.qc[l]);
      A.K = B(Ly.kv[l]);
      A.V = B(Ly.kv[l]);
      A.O = F(Ly.oc[l]);
      A.lse = F(Ly.lsec[l]);
      A.dsum = F(Ly.dsum);
      A.dO = F(Ly.tf);
      A.dQ = B(Ly.tb);
      A.dK = B(Ly.dkvb);
      A.dV = B(Ly.dkvb);
      A.zoff = (const int32_t*)(w + Ly.zoff);
      A.kv_cap = P.Pzt;
      A.ldq = d;
      A.ldkv = 2 * d;
      A.ldo = d;
      A.lddq = d;
      A.lddkv = 2 * d;
      A.kcol = 0;
      A.vcol = (int32_t)d;
      A.dkcol = 0;
      A.dvcol = (int32_t)d;
      A.Lq = S.chunk;
      A.max_lk = p->max_seqlen;
      A.hd = (int32_t)(d / H);
      A.nheads = (int32_t)H;
      A.scale = scale;
      attn(A, true);
    }
    wgrad_rows(B(Ly.tb), d, B(Ly.h2[l]), d, Gl(l, &jn_expert_layer_grads::wq_c), false);
    dgrad_rows(EPI_F32, B(Ly.tb), d, [&](int32_t g) { return ex[g].layers[l].wq_c; }, d, F(Ly.tf), true);
    wgrad_rows(B(Ly.dkvb), 2 * d, B(Ly.z), dp, Gl(l, &jn_expert_layer_grads::wkv_c), true);
    rms_bwd(Ly.x2[l], g2, ptr_table([&](int32_t g) { return (const void*)io[g].layers[l].g2; }));
    // self-attention block
    rows_copy(F(Ly.dx), false, B(Ly.dxb), true, P.Na, d);
    wgrad_rows(B(Ly.dxb), d, B(Ly.osb[l]), d, Gl(l, &jn_expert_layer_grads::wo_s), false);
    dgrad_rows(EPI_F32, B(Ly.dxb), d, [&](int32_t g) { return ex[g].layers[l].wo_s; }, d, F(Ly.tf), true);
    {
      AttnArgs A{};
      A.Q = B(Ly.qkv[l]);
      A.K = B(Ly.qkv[l]);
      A.V = B(Ly.qkv[l]);
      A.O = F(Ly.os[l]);
      A.lse = F(Ly.lses[l]);
      A.dsum = F(Ly.dsum);
      A.dO = F(Ly.tf);
      A.dQ = B(Ly.tb);
      A.dK = B(Ly.tb);
      A.dV = B(Ly.tb);
      A.ldq = 3 * d;
      A.ldkv = 3 * d;
      A.ldo = d;
      A.lddq = 3 * d;
      A.lddkv = 3 * d;
      A.kcol = (int32_t)d;
      A.vcol = (int32_t)(2 * d);
      A.dkcol = (int32_t)d;
      A.dvcol = (int32_t)(2 * d);
      A.Lq = S.chunk;
      A.max_lk = S.chunk;
      A.hd = (int32_t)(d / H);
      A.nheads = (int32_t)H;
      A.scale = scale;
      attn(A, true);
    }
    wgrad_rows(B(Ly.tb), 3 * d, B(Ly.h1[l]), d, Gl(l, &jn_expert_layer_grads::wqkv_s), false);
    dgrad_rows(EPI_F32, B(Ly.tb), 3 * d, [&](int32_t g) { return ex[g].layers[l].wqkv_s; }, d, F(Ly.tf), true);
    rms_bwd(Ly.x1[l], g1, ptr_table([&](int32_t g) { return (const void*)io[g].layers[l].g1; }));
  }
  // input projection and the padded output-projection gradient
  rows_copy(F(Ly.dx), false, B(Ly.dxb), true, P.Na, d);
  wgrad_rows(B(Ly.dxb), d, B(Ly.ub), KI, [&](int32_t g) { return F(Ly.dwinp) + (int64_t)g * d * KI; }, false);
  {
    std::vector<CopyDesc> v;
    for (int32_t g = 0; g < G; ++g) {
      const int32_t a = ex[g].action_dim;
      v.push_back(CopyDesc{F(Ly.dwinp) + (int64_t)g * d * KI, io[g].dw_in, KI, a, (int32_t)d, a, (int32_t)d, a, 0, 0, 0,
                           0});
      if (flow)
        v.push_back(CopyDesc{F(Ly.dwinp) + (int64_t)g * d * KI + kAP, io[g].dw_time, KI, S.dt, (int32_t)d, S.dt,
                             (int32_t)d, S.dt, 0, 0, 0, 0});
      v.push_back(CopyDesc{F(Ly.dwoutp) + (int64_t)g * kAP * d, io[g].dw_out, d, d, a, (int32_t)d, a, (int32_t)d, 0, 0, 0,
                           0});
    }
    copy(v);
  }
  if (rec.overflow) return fail(c, JN_ENOSPACE, "internal: expert descriptor arena too small");
  if (rec.bad_gemm) return fail(c, JN_EUNSUPPORTED, "internal: an expert GEMM has an unsupported shape");

  // ---- one upload of every table, then the launches in order
  st = stage_copy(c, darena, rec.img.data(), rec.img.size());
  if (st != JN_OK) return st;
  for (size_t i = 0; i < rec.ops.size(); ++i) {
    auto& op = rec.ops[i];
    JN_TRACED(c, rec.opcode[i], P.Na, d, 0, op(darena), "expert launch");
  }
  return JN_OK;
}

}  // extern "C"

// ------------------------------------------------------------ optimizer ---

namespace {

jn_status adamw_check(jn_ctx* c, const jn_adamw_tenant* t, int32_t G, int32_t* ntensors) {
  if (!t || G < 1) return fail(c, JN_EINVAL, "null tenants or G < 1");
  int64_t n = 0;
  auto aligned = [](const void* q) { return q && ((uintptr_t)q) % 16 == 0; };
  for (int32_t g = 0; g < G; ++g) {
    const jn_adamw_tenant& T = t[g];
    if (T.n_tensors < 0) return fail(c, JN_EINVAL, "tenant %d: n_tensors < 0", g);
    if (T.step < 1) return fail(c, JN_EINVAL, "tenant %d: step %lld < 1", g, (long long)T.step);
    if (!(T.lr >= 0.f) || !(T.beta1 >= 0.f && T.beta1 < 1.f) || !(T.beta2 >= 0.f && T.beta2 < 1.f) ||
        !(T.eps > 0.f) || !(T.weight_decay >= 0.f))
      return fail(c, JN_EINVAL, "tenant %d: hyperparameters out of range", g);
    if (T.n_tensors > 0 && (!T.params || !T.grads || !T.m || !T.v || !T.numel))
      return fail(c, JN_EINVAL, "tenant %d: null table", g);
    for (int32_t i = 0; i < T.n_tensors; ++i) {
      if (T.numel[i] < 0) return fail(c, JN_EINVAL, "tenant %d tensor %d: numel < 0", g, i);
      if (T.numel[i] == 0) continue;
      if (!aligned(T.params[i]) || !aligned(T.grads[i]) || !aligned(T.m[i]) || !aligned(T.v[i]))
        return fail(c, JN_EINVAL, "tenant %d tensor %d: null or unaligned pointer", g, i);
      if (T.bf16_out && T.bf16_out[i] && ((uintptr_t)T.bf16_out[i]) % 8 != 0)
        return fail(c, JN_EINVAL, "tenant %d tensor %d: bf16 copy not 8-byte aligned", g, i);
      if ((T.numel[i] + kAdamwBlockElems - 1) / kAdamwBlockElems >= (1ll << 30))
        return fail(c, JN_ESHAPE, "tenant %d tensor %d too large", g, i);
    }
    n += T.n_tensors;
  }
  if (n >= (1 << 24)) return fail(c, JN_ESHAPE, "too many tensors");
  *ntensors = (int32_t)n;
  return JN_OK;
}

size_t adamw_ws(int32_t n, int32_t G) {
  return align_up(sizeof(AdamwTensor) * (size_t)std::max(n, 1), 256) + align_up(sizeof(AdamwTenant) * G, 256);
}

}  // namespace

extern "C" {

jn_status jn_adamw_workspace_size(const jn_adamw_tenant* t, int32_t G, size_t* bytes) {
  if (!bytes) return JN_EINVAL;
  int32_t n = 0;
  jn_status st = adamw_check(nullptr, t, G, &n);
  if (st != JN_OK) return st;
  *bytes = adamw_ws(n, G);
  return JN_OK;
}

jn_status jn_tenant_adamw_step(jn_ctx* c, const jn_adamw_tenant* t, int32_t G, void* ws, size_t ws_bytes) {
  if (!c) return JN_EINVAL;
  int32_t n = 0;
  jn_status st = adamw_check(c, t, G, &n);
  if (st != JN_OK) return st;
  if (!ws || ((uintptr_t)ws) % 256 != 0) return fail(c, JN_EINVAL, "workspace null or not 256-byte aligned");
  const size_t need = adamw_ws(n, G);
  if (ws_bytes < need) return fail(c, JN_ENOSPACE, "workspace %zu B < %zu B", ws_bytes, need);
  const size_t ten_off = align_up(sizeof(AdamwTensor) * (size_t)std::max(n, 1), 256);
  std::vector<char> img(need, 0);
  AdamwTensor* tt = reinterpret_cast<AdamwTensor*>(img.data());
  AdamwTenant* th = reinterpret_cast<AdamwTenant*>(img.data() + ten_off);
  int32_t k = 0;
  for (int32_t g = 0; g < G; ++g) {
    const jn_adamw_tenant& T = t[g];
    const double bc1 = 1.0 - std::pow((double)T.beta1, (double)T.step);
    const double bc2 = 1.0 - std::pow((double)T.beta2, (double)T.step);
    th[g] = AdamwTenant{(float)(1.0 - (double)T.lr * T.weight_decay), (float)(T.lr / bc1), (float)(1.0 / std::sqrt(bc2)),
                        T.eps, T.beta1, T.beta2, 0.f, 0.f};
    for (int32_t i = 0; i < T.n_tensors; ++i, ++k) {
      tt[k] = AdamwTensor{T.params[i], T.grads[i], T.m[i], T.v[i],
                          (uint16_t*)(T.bf16_out ? T.bf16_out[i] : nullptr), T.numel[i], g, 0};
    }
  }
  const int32_t blocks = adamw_prepare(tt, n);
  if (blocks == 0) return JN_OK;
  st = stage_copy(c, ws, img.data(), need);
  if (st != JN_OK) return st;
  char* w = (char*)ws;
  JN_TRACED(c, JN_OP_OPTIMIZER, n, G, 0,
            launch_adamw(c->stream, (const AdamwTensor*)w, n, (const AdamwTenant*)(w + ten_off), blocks),
            "adamw kernel");
  return JN_OK;
}

}  // extern "C"

// ============================================================ inference ===
// Inference-side group batching (App. A.3 "Inference Queue Composition").
// The collector holds host metadata of queued requests in arrival order and
// releases the largest FIFO prefix that is compatible at the shared-prefix
// boundary, bounded by a maximum batch size and a timeout.  The plan makes
// one physical batch resident: every map and descriptor is uploaded once at
// creation, and a launch only enqueues kernels (pack, backbone, pool, head
// forward), which is what a HIP graph can record and replay.

struct jn_collector {
  struct Item {
    int64_t id;
    uint64_t sig;
    int32_t d, n;
    int64_t arrival;
  };
  int32_t max_batch = 0;
  int64_t timeout_us = 0;
  std::deque<Item> q;
};

struct jn_infer_plan {
  jn_packed packed{};
  std::vector<jn_layer> layers;
  jn_backbone bb{};
  void* hidden = nullptr;
  void* bb_ws = nullptr;
  size_t bb_bytes = 0;
  float* P = nullptr;
  const HeadGemm* dd = nullptr;
  const HeadTile* dt = nullptr;
  std::vector<std::pair<int32_t, int32_t>> fwd_rng, fwd_red;
  int32_t max_rows = 0;
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
};

namespace {

// Prefix the collector would release now: count of requests and whether the
// prefix can no longer grow (size reached, or the next queued request is
// incompatible or would overflow the batch).
void collector_prefix(const jn_collector* c, int32_t* count, int64_t* samples, bool* final_) {
  *count = 0;
  *samples = 0;
  *final_ = false;
  if (c->q.empty()) return;
  const jn_collector::Item& head = c->q.front();
  int64_t total = 0;
  int32_t k = 0;
  for (const jn_collector::Item& it : c->q) {
    if (it.sig != head.sig || it.d != head.d) {
      *final_ = true;
      break;
    }
    if (k > 0 && total + it.n > c->max_batch) {
      *final_ = true;
      break;
    }
    total += it.n;
    ++k;
    if (total >= c->max_batch) {
      *final_ = true;
      break;
    }
  }
  *count = k;
  *samples = total;
}

// Forward-only head plan inside `w` (fwd tables only): P | Z_k | H_k | split-K
// partials | descs | tiles.  A tenant's last layer writes the caller's action
// buffer (rows from 0) and is never split.
struct HeadFwdLayout {
  int maxL = 0;
  std::vector<int64_t> width;
  size_t P = 0, part = 0, descs = 0, tiles = 0, total = 0;
  std::vector<size_t> Z, H;
};

HeadFwdLayout head_fwd_layout(int64_t N, int64_t rows_bound, int64_t d, const jn_head* heads, int32_t G) {
  HeadFwdLayout L;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align_up(o + bytes, 256);
    return at;
  };
  for (int32_t g = 0; g < G; ++g) L.maxL = std::max(L.maxL, heads[g].n_layers);
  L.width.assign(L.maxL, 0);
  for (int32_t g = 0; g < G; ++g)
    for (int k = 0; k < heads[g].n_layers; ++k) L.width[k] = std::max<int64_t>(L.width[k], heads[g].dims[k + 1]);
  L.P = take(4 * N * d);
  L.Z.resize(L.maxL);
  L.H.resize(L.maxL);
  for (int k = 0; k < L.maxL; ++k) {
    L.Z[k] = take(4 * N * L.width[k]);
    L.H[k] = take(4 * N * L.width[k]);
  }
  const int64_t tm_dyn = (rows_bound + kHTM - 1) / kHTM;
  int64_t ntiles = 0, ndesc = 0, part_elems = 0;
  for (int32_t g = 0; g < G; ++g)
    for (int k = 0; k < heads[g].n_layers; ++k) {
      const int64_t sk = k + 1 < heads[g].n_layers ? head_ksplit(heads[g].dims[k]) : 1;
      ntiles += tm_dyn * ((heads[g].dims[k + 1] + kHTN - 1) / kHTN) * (sk + (sk > 1));
      if (sk > 1) part_elems = std::max(part_elems, sk * N * L.width[k]);
      ++ndesc;
    }
  L.part = take(4 * part_elems);
  L.descs = take(sizeof(HeadGemm) * ndesc);
  L.tiles = take(sizeof(HeadTile) * ntiles);
  L.total = o;
  return L;
}

// The plan's workspace: maps | tokens | hidden | backbone workspace | heads.
struct InferLayout {
  MapLayout m;
  BbLayout bl;
  HeadFwdLayout hl;
  size_t maps = 0, tokens = 0, hidden = 0, bb = 0, heads = 0, total = 0;
};

jn_status infer_layout(jn_ctx* c, const jn_request* req, int32_t R, const jn_tenant* ten, int32_t G,
                       const jn_pack_opts* o, const jn_backbone* bb, const jn_head* heads, Plan* p,
                       InferLayout* L) {
  jn_status st = make_plan(c, req, R, ten, G, o, p);
  if (st != JN_OK) return st;
  st = check_backbone(c, bb);
  if (st != JN_OK) return st;
  if (bb->d != o->d_model) return fail(c, JN_EINCOMPAT, "pack width %d != backbone width %d", o->d_model, bb->d);
  if (o->d_model % 8 != 0) return fail(c, JN_EUNSUPPORTED, "d_model %d not a multiple of 8", o->d_model);
  jn_packed shape{};
  shape.R = R;
  shape.G = G;
  shape.N = p->N;
  shape.T = p->T;
  shape.d = o->d_model;
  if (!heads) return fail(c, JN_EINVAL, "null heads");
  for (int32_t g = 0; g < G; ++g) {
    const jn_head& H = heads[g];
    if (H.n_layers < 1 || !H.dims || !H.W || !H.b) return fail(c, JN_EINVAL, "head %d incomplete", g);
    if (H.dims[0] != o->d_model) return fail(c, JN_EINCOMPAT, "head %d input %d != feature width %d", g, H.dims[0], o->d_model);
    for (int k = 0; k <= H.n_layers; ++k)
      if (H.dims[k] < 1) return fail(c, JN_EINVAL, "head %d dims[%d] < 1", g, k);
    if ((int64_t)H.action_dim * H.chunk != H.dims[H.n_layers])
      return fail(c, JN_EINVAL, "head %d output %d != action_dim*chunk", g, H.dims[H.n_layers]);
    for (int k = 0; k < H.n_layers; ++k)
      if (!H.W[k] || !H.b[k]) return fail(c, JN_EINVAL, "head %d layer %d null weight", g, k);
  }
  L->m = map_layout(p->N, p->T, G, R);
  L->bl = bb_layout(bb, p->T);
  int32_t max_n = 0;
  for (int32_t g = 0; g < G; ++g) max_n = std::max(max_n, p->toff[g + 1] - p->toff[g]);
  L->hl = head_fwd_layout(p->N, max_n, o->d_model, heads, G);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off = align_up(off + bytes, 256);
    return at;
  };
  L->maps = take(L->m.total);
  L->tokens = take((size_t)p->T * o->d_model * 2);
  L->hidden = take((size_t)p->T * o->d_model * 2);
  L->bb = take(L->bl.total);
  L->heads = take(L->hl.total);
  L->total = off;
  return JN_OK;
}

jn_status infer_enqueue(jn_ctx* c, const jn_infer_plan* pl) {
  const jn_packed& pk = pl->packed;
  hipStream_t s = c->stream;
  JN_TRACED(c, JN_OP_PACK, pk.T, pk.d, 0,
            launch_pack(s, (const ReqEntry*)pk.req_table, pk.sample_request, pk.sample_local, pk.seqlens,
                        pk.cu_seqlens, pk.N, pk.d, pk.align, pl->max_rows, pk.tokens, pk.token_sample,
                        pk.token_pos),
            "pack kernel");
  jn_status st = jn_backbone_forward(c, &pl->bb, &pk, pl->hidden, pl->bb_ws, pl->bb_bytes);
  if (st != JN_OK) return st;
  JN_TRACED(c, JN_OP_POOL, pk.T, pk.d, pk.N,
            launch_pool(s, pl->hidden, pk.seqlens, pk.cu_seqlens, pk.sample_tenant_rank, pk.N, pk.d, pl->P), "pool");
  for (size_t i = 0; i < pl->fwd_rng.size(); ++i) {
    const auto r = pl->fwd_rng[i], q = pl->fwd_red[i];
    if (r.second)
      JN_TRACED(c, JN_OP_HEAD_FWD, r.second, 0, 0,
                launch_head_gemm(s, pl->dd, pl->dt + r.first, r.second, pk.tenant_sample_off), "head fwd");
    if (q.second)
      JN_TRACED(c, JN_OP_HEAD_FWD, q.second, 0, 0,
                launch_head_reduce(s, pl->dd, pl->dt + q.first, q.second, pk.tenant_sample_off), "head fwd reduce");
  }
  return JN_OK;
}

}  // namespace

extern "C" {

jn_status jn_collector_create(jn_collector** out, int32_t max_batch_samples, int64_t timeout_us) {
  if (!out) return JN_EINVAL;
  *out = nullptr;
  if (max_batch_samples < 1 || timeout_us < 0) return JN_EINVAL;
  jn_collector* c = new (std::nothrow) jn_collector();
  if (!c) return JN_EINVAL;
  c->max_batch = max_batch_samples;
  c->timeout_us = timeout_us;
  *out = c;
  return JN_OK;
}

void jn_collector_destroy(jn_collector* c) { delete c; }

jn_status jn_collector_submit(jn_collector* c, int64_t request_id, uint64_t prefix_sig, int32_t d_model,
                              int32_t n_samples, int64_t arrival_us) {
  if (!c || n_samples < 1 || d_model < 1) return JN_EINVAL;
  if (!c->q.empty() && arrival_us < c->q.back().arrival) return JN_EINVAL;  // arrival order
  c->q.push_back(jn_collector::Item{request_id, prefix_sig, d_model, n_samples, arrival_us});
  return JN_OK;
}

jn_status jn_collector_poll(jn_collector* c, int64_t now_us, int64_t* ids, int32_t cap, int32_t* n) {
  if (!c || !n || (cap > 0 && !ids)) return JN_EINVAL;
  *n = 0;
  if (c->q.empty()) return JN_OK;
  int32_t k;
  int64_t samples;
  bool fin;
  collector_prefix(c, &k, &samples, &fin);
  const bool expired = now_us - c->q.front().arrival >= c->timeout_us;
  if (!fin && !expired) return JN_OK;
  if (cap < k) return JN_ENOSPACE;
  for (int32_t i = 0; i < k; ++i) {
    ids[i] = c->q.front().id;
    c->q.pop_front();
  }
  *n = k;
  return JN_OK;
}

jn_status jn_collector_status(const jn_collector* c, int32_t* pending, int64_t* deadline_us) {
  if (!c || !pending || !deadline_us) return JN_EINVAL;
  *pending = (int32_t)c->q.size();
  if (c->q.empty()) {
    *deadline_us = -1;
    return JN_OK;
  }
  int32_t k;
  int64_t samples;
  bool fin;
  collector_prefix(c, &k, &samples, &fin);
  *deadline_us = fin ? c->q.front().arrival : c->q.front().arrival + c->timeout_us;
  return JN_OK;
}

jn_status jn_infer_workspace_size(const jn_request* req, int32_t R, const jn_tenant* ten, int32_t G,
                                  const jn_pack_opts* o, const jn_backbone* bb, const jn_head* heads,
                                  size_t* bytes) {
  if (!bytes) return JN_EINVAL;
  Plan p;
  InferLayout L;
  jn_status st = infer_layout(nullptr, req, R, ten, G, o, bb, heads, &p, &L);
  if (st != JN_OK) return st;
  *bytes = L.total;
  return JN_OK;
}

jn_status jn_infer_plan_create(jn_ctx* c, const jn_request* req, int32_t R, const jn_tenant* ten, int32_t G,
                               const jn_pack_opts* o, const jn_backbone* bb, const jn_head* heads,
                               float* const* actions, void* ws, size_t ws_bytes, jn_infer_plan** out) {
  if (!c) return JN_EINVAL;
  if (!out || !actions || !ws) return fail(c, JN_EINVAL, "null output, actions or workspace");
  *out = nullptr;
  Plan p;
  InferLayout L;
  jn_status st = infer_layout(c, req, R, ten, G, o, bb, heads, &p, &L);
  if (st != JN_OK) return st;
  if (ws_bytes < L.total) return fail(c, JN_ENOSPACE, "workspace %zu B < %zu B", ws_bytes, L.total);
  if (((uintptr_t)ws) % 256 != 0) return fail(c, JN_EUNSUPPORTED, "workspace must be 256-byte aligned");
  if ((int64_t)p.N * ((o->d_model + 63) / 64) > 0x7fffffff) return fail(c, JN_ESHAPE, "too many samples for the pool grid");
  for (int32_t r = 0; r < R; ++r)
    if (((uintptr_t)req[r].embeds) % 16 != 0) return fail(c, JN_EUNSUPPORTED, "request %d embeds not 16-byte aligned", r);
  for (int32_t g = 0; g < G; ++g)
    if (!actions[g]) return fail(c, JN_EINVAL, "actions %d is null", g);

  jn_infer_plan* pl = new (std::nothrow) jn_infer_plan();
  if (!pl) return fail(c, JN_EINVAL, "out of host memory");
  char* w = (char*)ws;
  char* maps = w + L.maps;
  fill_packed(&pl->packed, maps, L.m, p, R, G, o);
  pl->packed.req_sig = request_signature(req, R);
  pl->packed.tokens = w + L.tokens;
  pl->max_rows = p.max_rows;
  pl->layers.assign(bb->layers, bb->layers + bb->n_layers);
  pl->bb = *bb;
  pl->bb.layers = pl->layers.data();
  pl->hidden = w + L.hidden;
  pl->bb_ws = w + L.bb;
  pl->bb_bytes = L.bl.total;

  // head forward descriptors: one launch per layer index, the last layer of
  // tenant g writing straight into actions[g] (rows in the tenant's arrival order)
  const HeadFwdLayout& hl = L.hl;
  char* hw = w + L.heads;
  pl->P = (float*)(hw + hl.P);
  const int64_t N = p.N, d = o->d_model;
  const int32_t tm_dyn = (int32_t)((tenant_rows_bound(&pl->packed) + kHTM - 1) / kHTM);
  std::vector<HeadGemm> descs;
  std::vector<HeadTile> tiles;
  for (int k = 0; k < hl.maxL; ++k) {
    int32_t t0 = (int32_t)tiles.size();
    for (int32_t g = 0; g < G; ++g) {
      const jn_head& Hh = heads[g];
      if (k >= Hh.n_layers) continue;
      const int64_t in = Hh.dims[k], outw = Hh.dims[k + 1];
      const bool last = k + 1 == Hh.n_layers;
      HeadGemm D{};
      D.A = (k == 0) ? pl->P : (const float*)(hw + hl.H[k - 1]);
      D.sam = (k == 0) ? d : hl.width[k - 1];
      D.sak = 1;
      D.B = Hh.W[k];
      D.sbk = 1;
      D.sbn = in;
      D.C = last ? actions[g] : (float*)(hw + hl.Z[k]);
      D.ldc = last ? outw : hl.width[k];
      D.bias = Hh.b[k];
      D.Cact = last ? nullptr : (float*)(hw + hl.H[k]);
      D.bumpA = D.sam;
      D.bumpB = 0;
      D.bumpC = last ? 0 : hl.width[k];
      D.M = -1;
      D.N = (int32_t)outw;
      D.K = (int32_t)in;
      D.tenant = g;
      D.tiles_n = (int32_t)((outw + kHTN - 1) / kHTN);
      D.ksplit = last ? 1 : head_ksplit(in);
      if (D.ksplit > 1) {
        D.part = (float*)(hw + hl.part);
        D.part_plane = N * hl.width[k];
      }
      const int32_t di = (int32_t)descs.size();
      descs.push_back(D);
      for (int32_t tk = 0; tk < D.ksplit; ++tk)
        for (int32_t tm = 0; tm < tm_dyn; ++tm)
          for (int32_t tn = 0; tn < D.tiles_n; ++tn) tiles.push_back(HeadTile{di, tm, tn, tk});
    }
    pl->fwd_rng.emplace_back(t0, (int32_t)tiles.size() - t0);
    const int32_t t1 = (int32_t)tiles.size();
    for (int32_t t = t0; t < t1; ++t)
      if (descs[tiles[t].desc].ksplit > 1 && tiles[t].tk == 0) tiles.push_back(tiles[t]);
    pl->fwd_red.emplace_back(t1, (int32_t)tiles.size() - t1);
  }
  const size_t dbytes = sizeof(HeadGemm) * descs.size(), tbytes = sizeof(HeadTile) * tiles.size();
  if (hl.descs + dbytes > hl.tiles || hl.tiles + tbytes > hl.total) {
    delete pl;
    return fail(c, JN_ENOSPACE, "internal: head table sizing");
  }
  pl->dd = (const HeadGemm*)(hw + hl.descs);
  pl->dt = (const HeadTile*)(hw + hl.tiles);

  // one-time uploads: maps, request table, head tables
  std::vector<char> img = host_head_image(L.m, p);
  std::vector<ReqEntry> rt(R);
  for (int32_t r = 0; r < R; ++r) rt[r] = ReqEntry{req[r].embeds, nullptr, req[r].max_len, req[r].n_samples, p.req_first[r], 0};
  std::vector<char> himg(hl.total - hl.descs, 0);
  std::memcpy(himg.data(), descs.data(), dbytes);
  std::memcpy(himg.data() + (hl.tiles - hl.descs), tiles.data(), tbytes);
  st = stage_copy(c, maps, img.data(), img.size());
  if (st == JN_OK) st = stage_copy(c, maps + L.m.reqtab, rt.data(), sizeof(ReqEntry) * R);
  if (st == JN_OK) st = stage_copy(c, hw + hl.descs, himg.data(), hl.tiles - hl.descs + tbytes);
  if (st != JN_OK) {
    delete pl;
    return st;
  }
  *out = pl;
  return JN_OK;
}

jn_status jn_infer_plan_packed(const jn_infer_plan* pl, jn_packed* out, void** hidden) {
  if (!pl || !out) return JN_EINVAL;
  *out = pl->packed;
  if (hidden) *hidden = pl->hidden;
  return JN_OK;
}

jn_status jn_infer_plan_launch(jn_ctx* c, const jn_infer_plan* pl) {
  if (!c) return JN_EINVAL;
  if (!pl) return fail(c, JN_EINVAL, "null plan");
  return infer_enqueue(c, pl);
}

jn_status jn_infer_plan_capture(jn_ctx* c, jn_infer_plan* pl) {
  if (!c) return JN_EINVAL;
  if (!pl) return fail(c, JN_EINVAL, "null plan");
  if (!c->stream) return fail(c, JN_EUNSUPPORTED, "graph capture needs a non-null stream");
  if (c->trace) return fail(c, JN_EUNSUPPORTED, "disable the launch trace before capturing");
  if (pl->exec) {
    hipGraphExecDestroy(pl->exec);
    pl->exec = nullptr;
  }
  if (pl->graph) {
    hipGraphDestroy(pl->graph);
    pl->graph = nullptr;
  }
  JN_HIP(c, hipStreamBeginCapture(c->stream, hipStreamCaptureModeThreadLocal), "hipStreamBeginCapture");
  jn_status st = infer_enqueue(c, pl);
  hipGraph_t graph = nullptr;
  hipError_t e = hipStreamEndCapture(c->stream, &graph);
  if (st != JN_OK) {
    if (graph) hipGraphDestroy(graph);
    return st;
  }
  if (e != hipSuccess || !graph) return hip_fail(c, e != hipSuccess ? e : hipErrorUnknown, "hipStreamEndCapture");
  hipGraphExec_t exec = nullptr;
  e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  if (e != hipSuccess) {
    hipGraphDestroy(graph);
    return hip_fail(c, e, "hipGraphInstantiate");
  }
  pl->graph = graph;
  pl->exec = exec;
  return JN_OK;
}

jn_status jn_infer_plan_replay(jn_ctx* c, const jn_infer_plan* pl) {
  if (!c) return JN_EINVAL;
  if (!pl || !pl->exec) return fail(c, JN_EINVAL, "plan has no captured graph");
  JN_HIP(c, hipGraphLaunch(pl->exec, c->stream), "hipGraphLaunch");
  return JN_OK;
}

void jn_infer_plan_destroy(jn_infer_plan* pl) {
  if (!pl) return;
  if (pl->exec) hipGraphExecDestroy(pl->exec);
  if (pl->graph) hipGraphDestroy(pl->graph);
  delete pl;
}

}  // extern "C"
