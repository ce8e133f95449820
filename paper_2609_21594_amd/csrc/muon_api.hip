// C ABI of the batched Muon step: argument checks, the shape-fused batch
// plan (Sec. 6.6), workspace and descriptor-table management, and the launch
// sequence per chunk.  Kernels live in muon_kernels.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstdint>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/muon_hip.h"
#include "muon_internal.h"

using muon::ChunkBuffers;
using muon::ChunkGeom;
using muon::MatDesc;
using muon::StepScalars;

// Event-pair timing of every launch (enabled on demand).
struct EventTimer : muon::LaunchTimer {
  struct Pending { int kind; hipEvent_t a, b; double flops, exec, bytes; };
  struct Acc { int64_t launches = 0; double ms = 0, flops = 0, exec = 0, bytes = 0; };
  std::vector<hipEvent_t> pool;
  std::vector<Pending> pending;
  Acc acc[muon::KK_COUNT];
  hipEvent_t cur_a = nullptr;
  bool failed = false;

  hipEvent_t take() {
    if (!pool.empty()) { hipEvent_t e = pool.back(); pool.pop_back(); return e; }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) { failed = true; return nullptr; }
    return e;
  }
  void begin(int, hipStream_t st) override {
    cur_a = take();
    if (cur_a && hipEventRecord(cur_a, st) != hipSuccess) failed = true;
  }
  void end(int kind, hipStream_t st, double flops, double exec, double bytes) override {
    hipEvent_t b = take();
    if (!cur_a || !b || hipEventRecord(b, st) != hipSuccess) { failed = true; return; }
    pending.push_back({kind, cur_a, b, flops, exec, bytes});
    cur_a = nullptr;
  }
  bool collect() {
    for (const Pending& p : pending) {
      float ms = 0.f;
      if (hipEventSynchronize(p.b) != hipSuccess || hipEventElapsedTime(&ms, p.a, p.b) != hipSuccess)
        failed = true;
      Acc& a = acc[p.kind];
      a.launches += 1; a.ms += ms; a.flops += p.flops; a.exec += p.exec; a.bytes += p.bytes;
      pool.push_back(p.a);
      pool.push_back(p.b);
    }
    pending.clear();
    return !failed;
  }
  void reset() { for (Acc& a : acc) a = Acc(); failed = false; }
  void destroy() {
    collect();
    for (hipEvent_t e : pool) (void)hipEventDestroy(e);
    pool.clear();
  }
};

// A descriptor table in device memory, filled from pinned staging memory.
struct DeviceTable {
  void* dev = nullptr;               // device copy
  size_t dev_cap = 0;                // bytes
  void* host = nullptr;              // pinned staging for the upload
  size_t host_cap = 0;
  hipEvent_t staged = nullptr;       // the last upload out of `host` has completed
  bool pending = false;
  std::vector<char> last;            // content of `dev`
};

struct CallCache;

struct muon_handle {
  int device = 0;
  bool profiling = false;
  EventTimer timer;
  void* ws = nullptr;
  size_t ws_bytes = 0;
  size_t ws_limit = 0;               // 0 = no cap
  DeviceTable mats;                  // MatDesc per matrix (muon_step, orthogonalize)
  DeviceTable adams;                 // AdamDesc per tensor (muon_adamw_step)
  // Every call's work uses the workspace and the tables; a call on another
  // stream than the previous one waits (on the device) for the previous
  // call's work first.
  hipEvent_t call_done = nullptr;
  hipStream_t last_stream = nullptr;
  bool have_last = false;
  // Chunk concurrency (muon_set_streams): chunks that leave CUs idle run on
  // a second stream with their own workspace slot, forked from and joined
  // back into the caller's stream through events.
  int nstreams = 2;
  // Grouped launches (muon_set_grouping): chunks that leave CUs idle and can
  // share a launch run each product of each step as one launch.
  int grouping = 1;
  hipStream_t side = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  bool log = false;                  // MUON_HIP_LOG set (and not "0"): each call's plan on stderr
  char err[512] = {0};               // message of the last failure (fixed: setting it allocates nothing)
  void* scratch = nullptr;           // this device's copy of the scratch array (see below), or null
  // The last request's validated form and plan, reused when the same request
  // comes again (see CallCache).
  CallCache* cache = nullptr;
};

namespace {

constexpr int64_t kDefaultChunkElems = int64_t(1) << 29;  // Sec. 6.6 batch cap
constexpr int kMaxSteps = 64;
constexpr int64_t kMaxDim = int64_t(1) << 28;
constexpr int64_t kMaxChunkMats = 65535;
const float kLegacyQuintic[3] = {3.4445f, -4.7750f, 2.0315f};

struct Msg {
  char* buf;
  size_t len;
  void set(const char* fmt, ...) {
    if (!buf || !len) return;
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, len, fmt, ap);
    va_end(ap);
  }
};

void set_err(muon_handle_t h, const char* fmt, ...) {
  if (!h) return;
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(h->err, sizeof h->err, fmt, ap);
  va_end(ap);
}

size_t dtype_size(int dt) { return dt == MUON_BF16 ? 2 : 4; }
bool dtype_ok(int dt) { return dt == MUON_F32 || dt == MUON_BF16; }

// One matrix of the request, before planning.  Row i of the matrix starts at
// element (i / rb)*bs + (i % rb)*ld of W, g and out, and (i / rb)*bs_b +
// (i % rb)*ld_b of buf.
struct Item {
  int64_t flat;            // entry-major, plane-minor index
  int64_t rows, cols;
  int32_t pdt, gdt;
  void* W; const void* g; float* buf; void* out;
  int64_t ld, rb, bs, ld_b, bs_b;
  int32_t cset;            // coefficient table (index into the call's table list)
  int32_t scale_mode;      // 0: 0.2 sqrt(max(m, n)); 1: none; 2: sqrt(max(1, m/n))
  double post_scale;       // factor applied to the updated matrix (1: none)
};

// The distinct coefficient tables of a call: [0] is the call's own table,
// then every per-entry table whose values differ from all earlier ones.
using CoeffTables = std::vector<std::vector<float>>;

std::vector<float> coefficient_table(int K, const float* coeffs);

int32_t table_id(CoeffTables& tables, std::vector<float> t) {
  for (size_t i = 0; i < tables.size(); ++i)
    if (tables[i] == t) return int32_t(i);
  tables.push_back(std::move(t));
  return int32_t(tables.size() - 1);
}

void set_dense(Item& it) {
  it.ld = it.ld_b = it.cols;
  it.rb = it.rows;
  it.bs = it.bs_b = it.rows * it.cols;
}

// A run of `count` equal byte intervals [lo + k*stride, lo + k*stride + len),
// k = 0..count-1, with stride >= len when count > 1 (the intervals of a run
// never overlap each other).  A buffer a call touches is a few runs: one
// interval when dense, one run over all its rows when rows, blocks and
// planes continue one stride (a column range of a contiguous tensor).
struct Run {
  uintptr_t lo, stride, len;
  int64_t count;
  bool written;
  uintptr_t hi() const { return lo + uintptr_t(count - 1) * stride + len; }  // end of the hull
};

int64_t floor_div(int64_t x, int64_t s) { return x >= 0 ? x / s : -((-x + s - 1) / s); }

// Does [x, x + len) meet an interval of run t?  The first interval of t that
// ends after x is the only candidate.
bool interval_meets(uintptr_t x, uintptr_t len, const Run& t) {
  if (x < t.lo + t.len) return t.lo < x + len;
  if (t.count == 1) return false;
  const int64_t j = int64_t((x - t.lo - t.len) / t.stride) + 1;
  return j < t.count && t.lo + uintptr_t(j) * t.stride < x + len;
}

// Exact intersection test of two runs whose hulls overlap.
bool runs_meet(const Run& a, const Run& b) {
  if (a.count == 1) return interval_meets(a.lo, a.len, b);
  if (b.count == 1) return interval_meets(b.lo, b.len, a);
  if (a.stride == b.stride) {
    // a_i meets b_j iff -b.len < D + (j - i)*s < a.len with D = b.lo - a.lo;
    // every q = j - i in [1 - a.count, b.count - 1] is reachable.
    const int64_t s = int64_t(a.stride), D = int64_t(b.lo) - int64_t(a.lo);
    const int64_t q_lo = std::max(floor_div(-int64_t(b.len) - D, s) + 1, 1 - a.count);
    const int64_t q_hi = std::min(-floor_div(D - int64_t(a.len), s) - 1, b.count - 1);
    return q_lo <= q_hi;
  }
  // different strides: walk the intervals of the run with fewer of them that
  // lie inside the other's hull
  const Run& w = a.count <= b.count ? a : b;
  const Run& o = a.count <= b.count ? b : a;
  const int64_t k0 = o.lo < w.lo + w.len ? 0 : int64_t((o.lo - w.lo - w.len) / w.stride) + 1;
  for (int64_t k = k0; k < w.count; ++k) {
    const uintptr_t x = w.lo + uintptr_t(k) * w.stride;
    if (x >= o.hi()) break;
    if (interval_meets(x, w.len, o)) return true;
  }
  return false;
}

// Written runs may not meet anything; read-only runs may meet each other.
// Exact in-place pairs (orthogonalize in[i] == out[i]) are passed in merged
// as one written run.  Runs are swept in order of their start; only runs
// whose hulls overlap are compared.
bool runs_disjoint(std::vector<Run>& rs) {
  std::sort(rs.begin(), rs.end(), [](const Run& a, const Run& b) { return a.lo < b.lo; });
  std::vector<const Run*> open;  // earlier runs whose hull reaches past the current start
  for (const Run& r : rs) {
    if (r.len == 0 || r.count == 0) continue;
    open.erase(std::remove_if(open.begin(), open.end(), [&](const Run* o) { return o->hi() <= r.lo; }),
               open.end());
    for (const Run* o : open)
      if ((o->written || r.written) && runs_meet(*o, r)) return false;
    open.push_back(&r);
  }
  return true;
}

muon_status_t check_hparams(const muon_hparams_t* hp, Msg& msg) {
  if (!hp) { msg.set("hparams is NULL"); return MUON_ERR_INVALID_ARGUMENT; }
  if (!std::isfinite(hp->lr) || !std::isfinite(hp->beta) || !std::isfinite(hp->weight_decay) ||
      !std::isfinite(hp->eps) || hp->eps < 0.f) {
    msg.set("lr, beta, weight_decay must be finite and eps finite and >= 0");
    return MUON_ERR_INVALID_ARGUMENT;
  }
  if (hp->ns_steps < 0 || hp->ns_steps > kMaxSteps) {
    msg.set("ns_steps must be in [0, %d]", kMaxSteps);
    return MUON_ERR_INVALID_ARGUMENT;
  }
  if (hp->nesterov != 0 && hp->nesterov != 1) { msg.set("nesterov must be 0 or 1"); return MUON_ERR_INVALID_ARGUMENT; }
  if (hp->ns_precision != MUON_NS_BF16 && hp->ns_precision != MUON_NS_F32) {
    msg.set("unknown ns_precision %d", int(hp->ns_precision));
    return MUON_ERR_INVALID_ARGUMENT;
  }
  if (hp->scale_mode < 0 || hp->scale_mode > 2) { msg.set("scale_mode must be 0, 1 or 2"); return MUON_ERR_INVALID_ARGUMENT; }
  if (hp->max_chunk_elems < 0) { msg.set("max_chunk_elems must be >= 0"); return MUON_ERR_INVALID_ARGUMENT; }
  if (hp->ns_coeffs)
    for (int i = 0; i < 3 * hp->ns_steps; ++i)
      if (!std::isfinite(hp->ns_coeffs[i])) { msg.set("ns_coeffs[%d] is not finite", i); return MUON_ERR_INVALID_ARGUMENT; }
  return MUON_OK;
}

muon_status_t check_dims(int64_t rows, int64_t cols, int64_t batch, const char* what, int64_t i, Msg& msg) {
  if (rows < 1 || cols < 1 || batch < 1) {
    msg.set("%s %lld: rows, cols and batch must be >= 1", what, (long long)i);
    return MUON_ERR_INVALID_ARGUMENT;
  }
  if (rows > kMaxDim || cols > kMaxDim) {
    msg.set("%s %lld: rows and cols must be <= 2^28", what, (long long)i);
    return MUON_ERR_UNSUPPORTED;
  }
  return MUON_OK;
}

// The first and one-past-last byte a buffer of a call touches.
struct Span { uintptr_t lo, hi; };

Span hull(const std::vector<Run>& rs, size_t from) {
  Span s{UINTPTR_MAX, 0};
  for (size_t i = from; i < rs.size(); ++i) {
    s.lo = std::min(s.lo, rs[i].lo);
    s.hi = std::max(s.hi, rs[i].hi());
  }
  return s;
}

// The bytes a view of `batch` planes occupies, as runs.  Row i of plane e
// starts at element e*ps + (i / rb)*bs + (i % rb)*ld; validation has already
// ensured that rows, blocks and planes follow each other without overlap.
// Levels (row, block, plane) merge inward while they are contiguous or
// continue the stride inside them; the innermost level left is the run, and
// one run is emitted per index of the levels outside it.
void view_runs(uintptr_t base, size_t es, int64_t rows, int64_t cols, int64_t batch, int64_t ld,
               int64_t rb, int64_t bs, int64_t ps, bool written, std::vector<Run>& out) {
  struct Level { int64_t stride, count; };
  const Level all[3] = {{ld, rb}, {bs, rows / rb}, {ps, batch}};
  Level lv[3];
  int n = 0;
  for (const Level& l : all)
    if (l.count > 1) lv[n++] = l;
  int64_t len = cols;
  for (bool merged = true; merged;) {
    merged = false;
    if (n > 0 && lv[0].stride == len) {  // contiguous: one longer interval
      len *= lv[0].count;
      std::copy(lv + 1, lv + n, lv);
      --n;
      merged = true;
      continue;
    }
    for (int i = 0; i + 1 < n && !merged; ++i)
      if (lv[i + 1].stride == lv[i].stride * lv[i].count) {  // continues the stride inside it
        lv[i].count *= lv[i + 1].count;
        std::copy(lv + i + 2, lv + n, lv + i + 1);
        --n;
        merged = true;
      }
  }
  const int64_t stride = n > 0 ? lv[0].stride : len, count = n > 0 ? lv[0].count : 1;
  const int64_t c1 = n > 1 ? lv[1].count : 1, s1 = n > 1 ? lv[1].stride : 0;
  const int64_t c2 = n > 2 ? lv[2].count : 1, s2 = n > 2 ? lv[2].stride : 0;
  for (int64_t p = 0; p < c2; ++p)
    for (int64_t q = 0; q < c1; ++q)
      out.push_back({base + uintptr_t(p * s2 + q * s1) * es, uintptr_t(stride) * es, uintptr_t(len) * es,
                     count, written});
}

muon_status_t validate_step(const muon_param_t* params, int64_t n, const muon_hparams_t* hp,
                            std::vector<Item>* items, CoeffTables* tables, Msg& msg,
                            std::vector<Span>* spans = nullptr) {
  muon_status_t st = check_hparams(hp, msg);
  if (st != MUON_OK) return st;
  if (tables) {
    tables->clear();
    tables->push_back(coefficient_table(hp->ns_steps, hp->ns_coeffs));
  }
  if (n < 0) { msg.set("n must be >= 0"); return MUON_ERR_INVALID_ARGUMENT; }
  if (n > 0 && !params) { msg.set("params is NULL"); return MUON_ERR_INVALID_ARGUMENT; }
  std::vector<Run> runs;
  runs.reserve(3 * n);
  int64_t flat = 0;
  for (int64_t i = 0; i < n; ++i) {
    const muon_param_t& p = params[i];
    if (!p.param || !p.grad || !p.momentum) { msg.set("entry %lld: NULL pointer", (long long)i); return MUON_ERR_INVALID_ARGUMENT; }
    if ((st = check_dims(p.rows, p.cols, p.batch, "entry", i, msg)) != MUON_OK) return st;
    if (!dtype_ok(p.param_dtype) || !dtype_ok(p.grad_dtype)) { msg.set("entry %lld: unknown dtype", (long long)i); return MUON_ERR_INVALID_ARGUMENT; }
    const int64_t plane = p.rows * p.cols;
    if (p.batch > (int64_t(1) << 40) / plane) { msg.set("entry %lld: too many elements", (long long)i); return MUON_ERR_UNSUPPORTED; }
    // the logical-matrix view (zero fields take their dense defaults)
    if (p.ld < 0 || p.row_block < 0 || p.block_stride < 0 || p.plane_stride < 0) {
      msg.set("entry %lld: negative stride", (long long)i);
      return MUON_ERR_INVALID_ARGUMENT;
    }
    if (p.momentum_dense != 0 && p.momentum_dense != 1) {
      msg.set("entry %lld: momentum_dense must be 0 or 1", (long long)i);
      return MUON_ERR_INVALID_ARGUMENT;
    }
    if (p.post_scale != 0.f && !(std::isfinite(p.post_scale) && p.post_scale > 0.f)) {
      msg.set("entry %lld: post_scale must be 0 (none) or finite and > 0", (long long)i);
      return MUON_ERR_INVALID_ARGUMENT;
    }
    const int64_t ld = p.ld ? p.ld : p.cols;
    const int64_t rb = p.row_block ? p.row_block : p.rows;
    if (ld < p.cols) { msg.set("entry %lld: ld < cols", (long long)i); return MUON_ERR_INVALID_ARGUMENT; }
    if (rb > p.rows || p.rows % rb) { msg.set("entry %lld: row_block must divide rows", (long long)i); return MUON_ERR_INVALID_ARGUMENT; }
    const int64_t nblk = p.rows / rb;
    // strides beyond 2^46 elements are refused before any product is formed
    constexpr int64_t kMaxStride = int64_t(1) << 46;
    if (ld > kMaxStride || p.block_stride > kMaxStride || p.plane_stride > kMaxStride) {
      msg.set("entry %lld: stride too large", (long long)i);
      return MUON_ERR_UNSUPPORTED;
    }
    const int64_t bs = p.block_stride ? p.block_stride : rb * ld;
    const double span_d = double(nblk - 1) * double(bs) + double(rb - 1) * double(ld) + double(p.cols);
    if (span_d > double(kMaxStride)) { msg.set("entry %lld: view too large", (long long)i); return MUON_ERR_UNSUPPORTED; }
    const int64_t span = (nblk - 1) * bs + (rb - 1) * ld + p.cols;  // elements one plane spans
    if (nblk > 1 && bs < (rb - 1) * ld + p.cols) {
      msg.set("entry %lld: row blocks overlap (block_stride too small)", (long long)i);
      return MUON_ERR_INVALID_ARGUMENT;
    }
    const int64_t ps = p.plane_stride ? p.plane_stride : nblk * bs;
    if (p.batch > 1 && ps < span) { msg.set("entry %lld: planes overlap (plane_stride too small)", (long long)i); return MUON_ERR_INVALID_ARGUMENT; }
    if (double(p.batch - 1) * double(ps) + double(span) > double(int64_t(1) << 48)) {
      msg.set("entry %lld: view too large", (long long)i);
      return MUON_ERR_UNSUPPORTED;
    }
    // per-parameter coefficient table and scale
    if (p.ns_coeffs) {
      if (p.ns_steps < 0 || p.ns_steps > kMaxSteps) {
        msg.set("entry %lld: ns_steps must be in [0, %d]", (long long)i, kMaxSteps);
        return MUON_ERR_INVALID_ARGUMENT;
      }
      for (int k = 0; k < 3 * p.ns_steps; ++k)
        if (!std::isfinite(p.ns_coeffs[k])) {
          msg.set("entry %lld: ns_coeffs[%d] is not finite", (long long)i, k);
          return MUON_ERR_INVALID_ARGUMENT;
        }
    }
    if (p.scale_mode < 0 || p.scale_mode > 3) {
      msg.set("entry %lld: scale_mode must be 0 (the call's) or 1 + a scale_mode", (long long)i);
      return MUON_ERR_INVALID_ARGUMENT;
    }
    int32_t cset = 0;
    if (tables && p.ns_coeffs)
      cset = table_id(*tables, std::vector<float>(p.ns_coeffs, p.ns_coeffs + 3 * p.ns_steps));
    const int32_t smode = p.scale_mode ? p.scale_mode - 1 : hp->scale_mode;
    const bool mdense = p.momentum_dense != 0;
    const uintptr_t W = reinterpret_cast<uintptr_t>(p.param), G = reinterpret_cast<uintptr_t>(p.grad),
                    M = reinterpret_cast<uintptr_t>(p.momentum);
    if ((W % dtype_size(p.param_dtype)) || (G % dtype_size(p.grad_dtype)) || (M % 4)) {
      msg.set("entry %lld: pointer not aligned to its element size", (long long)i);
      return MUON_ERR_INVALID_ARGUMENT;
    }
    const size_t r0 = runs.size();
    view_runs(W, dtype_size(p.param_dtype), p.rows, p.cols, p.batch, ld, rb, bs, ps, true, runs);
    const size_t r1 = runs.size();
    view_runs(G, dtype_size(p.grad_dtype), p.rows, p.cols, p.batch, ld, rb, bs, ps, false, runs);
    const size_t r2 = runs.size();
    if (mdense) view_runs(M, 4, p.rows, p.cols, p.batch, p.cols, p.rows, plane, plane, true, runs);
    else view_runs(M, 4, p.rows, p.cols, p.batch, ld, rb, bs, ps, true, runs);
    if (spans) {
      const std::vector<Run> w(runs.begin() + long(r0), runs.begin() + long(r1));
      const std::vector<Run> g(runs.begin() + long(r1), runs.begin() + long(r2));
      spans->push_back(hull(w, 0));
      spans->push_back(hull(g, 0));
      spans->push_back(hull(runs, r2));
    }
    if (items) {
      for (int64_t e = 0; e < p.batch; ++e) {
        Item it;
        it.flat = flat++;
        it.rows = p.rows; it.cols = p.cols;
        it.pdt = p.param_dtype; it.gdt = p.grad_dtype;
        it.W = static_cast<char*>(p.param) + e * ps * int64_t(dtype_size(p.param_dtype));
        it.g = static_cast<const char*>(p.grad) + e * ps * int64_t(dtype_size(p.grad_dtype));
        it.buf = p.momentum + (mdense ? e * plane : e * ps);
        it.out = nullptr;
        it.ld = ld; it.rb = rb; it.bs = bs;
        it.ld_b = mdense ? p.cols : ld;
        it.bs_b = mdense ? rb * p.cols : bs;
        it.cset = cset;
        it.scale_mode = smode;
        it.post_scale = p.post_scale != 0.f ? double(p.post_scale) : 1.0;
        // row blocks that follow each other at the row stride are no blocks
        if (it.bs == rb * it.ld && it.bs_b == rb * it.ld_b) {
          it.rb = p.rows;
          it.bs = p.rows * it.ld;
          it.bs_b = p.rows * it.ld_b;
        }
        items->push_back(it);
      }
    }
  }
  if (!runs_disjoint(runs)) {
    msg.set("param, grad and momentum buffers overlap");
    return MUON_ERR_INVALID_ARGUMENT;
  }
  return MUON_OK;
}

// The checks of ns_orthogonalize_batched that concern no single matrix.
muon_status_t check_orth_args(const void* const* in, void* const* out, const int64_t* rows,
                              const int64_t* cols, int64_t n, int dtype, int32_t ns_steps,
                              const float* coeffs, float eps, int prec, Msg& msg) {
  if (n < 0) { msg.set("n must be >= 0"); return MUON_ERR_INVALID_ARGUMENT; }
  if (n > 0 && (!in || !out || !rows || !cols)) { msg.set("NULL array argument"); return MUON_ERR_INVALID_ARGUMENT; }
  if (!dtype_ok(dtype)) { msg.set("unknown dtype"); return MUON_ERR_INVALID_ARGUMENT; }
  if (ns_steps < 0 || ns_steps > kMaxSteps) { msg.set("ns_steps must be in [0, %d]", kMaxSteps); return MUON_ERR_INVALID_ARGUMENT; }
  if (!std::isfinite(eps) || eps < 0.f) { msg.set("eps must be finite and >= 0"); return MUON_ERR_INVALID_ARGUMENT; }
  if (prec != MUON_NS_BF16 && prec != MUON_NS_F32) { msg.set("unknown ns precision"); return MUON_ERR_INVALID_ARGUMENT; }
  if (coeffs)
    for (int i = 0; i < 3 * ns_steps; ++i)
      if (!std::isfinite(coeffs[i])) { msg.set("ns_coeffs[%d] is not finite", i); return MUON_ERR_INVALID_ARGUMENT; }
  return MUON_OK;
}

// One matrix of ns_orthogonalize_batched: pointers, extents, alignment.
muon_status_t check_orth_matrix(const void* in, const void* out, int64_t rows, int64_t cols, size_t es,
                                int64_t i, Msg& msg) {
  if (!in || !out) { msg.set("matrix %lld: NULL pointer", (long long)i); return MUON_ERR_INVALID_ARGUMENT; }
  const muon_status_t st = check_dims(rows, cols, 1, "matrix", i, msg);
  if (st != MUON_OK) return st;
  if (reinterpret_cast<uintptr_t>(in) % es || reinterpret_cast<uintptr_t>(out) % es) {
    msg.set("matrix %lld: pointer not aligned to its element size", (long long)i);
    return MUON_ERR_INVALID_ARGUMENT;
  }
  return MUON_OK;
}

Item orth_item(const void* in, void* out, int64_t rows, int64_t cols, int dtype, int64_t i) {
  Item it{};
  it.flat = i; it.rows = rows; it.cols = cols;
  it.pdt = dtype; it.gdt = dtype;
  it.W = nullptr; it.g = in; it.buf = nullptr; it.out = out;
  set_dense(it);
  it.cset = 0;
  it.scale_mode = 1;
  it.post_scale = 1.0;
  return it;
}

muon_status_t validate_orth(const void* const* in, void* const* out, const int64_t* rows,
                            const int64_t* cols, int64_t n, int dtype, int32_t ns_steps,
                            const float* coeffs, float eps, int prec, std::vector<Item>* items,
                            Msg& msg, std::vector<Span>* spans = nullptr) {
  muon_status_t st = check_orth_args(in, out, rows, cols, n, dtype, ns_steps, coeffs, eps, prec, msg);
  if (st != MUON_OK) return st;
  std::vector<Run> runs;
  const size_t es = dtype_size(dtype);
  for (int64_t i = 0; i < n; ++i) {
    if ((st = check_orth_matrix(in[i], out[i], rows[i], cols[i], es, i, msg)) != MUON_OK) return st;
    const uintptr_t a = reinterpret_cast<uintptr_t>(in[i]), b = reinterpret_cast<uintptr_t>(out[i]);
    const uintptr_t bytes = uintptr_t(rows[i]) * uintptr_t(cols[i]) * es;
    if (a == b) {
      runs.push_back({a, bytes, bytes, 1, true});
    } else {
      runs.push_back({a, bytes, bytes, 1, false});
      runs.push_back({b, bytes, bytes, 1, true});
    }
    if (spans) {
      spans->push_back({a, a + bytes});
      if (b != a) spans->push_back({b, b + bytes});
    }
    if (items) items->push_back(orth_item(in[i], out[i], rows[i], cols[i], dtype, i));
  }
  if (!runs_disjoint(runs)) { msg.set("an output overlaps another buffer"); return MUON_ERR_INVALID_ARGUMENT; }
  return MUON_OK;
}

// ---------------------------------------------------------------------------
// Plan: bucket by (short side, long side, dtypes) after transpose-first,
// largest work first, chunks of at most `cap` elements (at least one matrix).
// ---------------------------------------------------------------------------
struct Chunk {
  int64_t s, l, S, L;
  int32_t pdt, gdt;
  int32_t cset;
  int64_t first, count;
  size_t bytes;
  // byte offsets inside the workspace
  size_t off_X[2], off_XT[2], off_A, off_B, off_part, off_r, off_sync;
  bool keeps_xt;  // X^T buffers present (see chunk_keeps_xt)
};

struct Plan {
  std::vector<int64_t> order;  // plan position -> index into items
  std::vector<Chunk> chunks;
  size_t ws_bytes = 0;
};

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// Workspace of a chunk of c.count matrices of padded extent c.S x c.L: two
// X buffers (and two X^T where kept), A, B, the fp64 norm partials, then r
// (fp64) and the first step's scale (fp32) per matrix; byte offsets and the
// total in c.
void layout_chunk(Chunk& c, bool ns_f32, int K) {
  const size_t es = ns_f32 ? 4 : 2;
  const size_t xb = align256(size_t(c.count) * size_t(c.S) * size_t(c.L) * es);
  const size_t ab = align256(size_t(c.count) * size_t(c.S) * size_t(c.S) * es);
  const bool small = muon::chunk_is_small(c.s, c.l, ns_f32);
  const size_t parts = std::max<size_t>(size_t(muon::norm_tiles(c.S, c.L)), small ? muon::kSmallMaxGroup : 0);
  const size_t pb = align256(size_t(c.count) * parts * 8);
  c.keeps_xt = muon::chunk_keeps_xt(c.S, c.L, ns_f32, K);
  size_t off = 0;
  c.off_X[0] = off; off += xb;
  c.off_X[1] = off; off += xb;
  if (c.keeps_xt) {
    c.off_XT[0] = off; off += xb;
    c.off_XT[1] = off; off += xb;
  }
  c.off_A = off; off += ab;
  c.off_B = off; off += ab;
  c.off_part = off; off += pb;
  c.off_r = off; off += align256(size_t(c.count) * 12);  // rscale (fp64), then xscale (fp32)
  c.off_sync = off; off += small ? size_t(muon::kSmallSyncBytes) : 0;
  c.bytes = off;
}

// `steps[c]` is the step count of coefficient table c; the work of a
// bucket is s^2 l per step (at least one, so K = 0 buckets keep their
// shape order).
Plan make_plan(const std::vector<Item>& items, int64_t cap, bool ns_f32, const std::vector<int>& steps) {
  if (cap <= 0) cap = kDefaultChunkElems;
  using Key = std::tuple<int64_t, int64_t, int32_t, int32_t, int32_t>;
  std::map<Key, std::vector<int64_t>> buckets;
  std::map<Key, int64_t> first_seen;
  for (size_t i = 0; i < items.size(); ++i) {
    const Item& it = items[i];
    Key k{std::min(it.rows, it.cols), std::max(it.rows, it.cols), it.pdt, it.gdt, it.cset};
    if (!first_seen.count(k)) first_seen[k] = int64_t(i);
    buckets[k].push_back(int64_t(i));
  }
  std::vector<Key> keys;
  for (auto& kv : buckets) keys.push_back(kv.first);
  auto work = [&](const Key& k) {
    return double(std::get<0>(k)) * std::get<0>(k) * std::get<1>(k) *
           std::max(1, steps[size_t(std::get<4>(k))]);
  };
  std::stable_sort(keys.begin(), keys.end(), [&](const Key& a, const Key& b) {
    const double wa = work(a), wb = work(b);
    if (wa != wb) return wa > wb;
    return first_seen[a] < first_seen[b];
  });
  Plan plan;
  for (const Key& k : keys) {
    const auto& idx = buckets[k];
    const int64_t s = std::get<0>(k), l = std::get<1>(k);
    const int64_t per = std::max<int64_t>(1, std::min<int64_t>(kMaxChunkMats, cap / (s * l)));
    for (size_t b = 0; b < idx.size(); b += size_t(per)) {
      Chunk c{};
      c.s = s; c.l = l;
      c.S = muon::round_up(s, muon::kPad);
      c.L = muon::round_up(l, muon::kPad);
      c.pdt = std::get<2>(k); c.gdt = std::get<3>(k);
      c.cset = std::get<4>(k);
      c.first = int64_t(plan.order.size());
      c.count = std::min<int64_t>(per, int64_t(idx.size() - b));
      for (int64_t j = 0; j < c.count; ++j) plan.order.push_back(idx[b + size_t(j)]);
      layout_chunk(c, ns_f32, steps[size_t(c.cset)]);
      plan.ws_bytes = std::max(plan.ws_bytes, c.bytes);
      plan.chunks.push_back(c);
    }
  }
  return plan;
}

struct DeviceGuard {
  int prev = -1;
  bool ok = false;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) return;
    ok = hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() { if (prev >= 0) (void)hipSetDevice(prev); }
};

muon_status_t device_fail(muon_handle_t h, const char* what, hipError_t e) {
  set_err(h, "%s: %s", what, hipGetErrorString(e));
  return MUON_ERR_DEVICE;
}

// Blocks until every call made on the handle has finished on the device.
// Each call records call_done at its end on its stream, after waiting for
// the previous call's call_done when it runs on another stream, so the last
// one covers all of them; unrelated work on the device is not waited for.
muon_status_t wait_idle(muon_handle_t h) {
  if (!h->have_last) return MUON_OK;
  const hipError_t e = hipEventSynchronize(h->call_done);
  return e == hipSuccess ? MUON_OK : device_fail(h, "hipEventSynchronize", e);
}

muon_status_t ensure_workspace(muon_handle_t h, size_t bytes) {
  if (bytes <= h->ws_bytes) return MUON_OK;
  if (h->ws_limit && bytes > h->ws_limit) {
    set_err(h, "workspace of %zu bytes exceeds the limit of %zu bytes", bytes, h->ws_limit);
    return MUON_ERR_OUT_OF_MEMORY;
  }
  hipError_t e;
  if (h->ws) {
    // earlier calls' work may still use the old workspace
    const muon_status_t st = wait_idle(h);
    if (st != MUON_OK) return st;
    if ((e = hipFree(h->ws)) != hipSuccess) return device_fail(h, "hipFree", e);
    h->ws = nullptr;
    h->ws_bytes = 0;
  }
  void* p = nullptr;
  e = hipMalloc(&p, bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    set_err(h, "hipMalloc of %zu workspace bytes failed: %s", bytes, hipGetErrorString(e));
    return MUON_ERR_OUT_OF_MEMORY;
  }
  h->ws = p;
  h->ws_bytes = bytes;
  return MUON_OK;
}

// Puts `bytes` bytes at `data` into t.dev on `stream`, skipping the copy
// when the device table already holds exactly these bytes.  The caller has
// ordered `stream` after every earlier call's work (begin_call).
muon_status_t upload_table(muon_handle_t h, DeviceTable& t, const void* data, size_t bytes,
                           hipStream_t stream) {
  if (bytes == t.last.size() && std::memcmp(data, t.last.data(), bytes) == 0) return MUON_OK;
  hipError_t e;
  if (bytes > t.dev_cap) {
    const size_t cap = std::max(bytes, size_t(16384));
    if (t.dev) {
      const muon_status_t st = wait_idle(h);  // earlier calls may still read the old table
      if (st != MUON_OK) return st;
      if ((e = hipFree(t.dev)) != hipSuccess) return device_fail(h, "hipFree", e);
      t.dev = nullptr; t.dev_cap = 0; t.last.clear();
    }
    if ((e = hipMalloc(&t.dev, cap)) != hipSuccess) {
      (void)hipGetLastError();
      set_err(h, "hipMalloc of a descriptor table failed");
      return MUON_ERR_OUT_OF_MEMORY;
    }
    t.dev_cap = cap;
  }
  if (t.pending) {
    if ((e = hipEventSynchronize(t.staged)) != hipSuccess) return device_fail(h, "hipEventSynchronize", e);
    t.pending = false;
  }
  if (bytes > t.host_cap) {
    if (t.host) { (void)hipHostFree(t.host); t.host = nullptr; t.host_cap = 0; }
    const size_t cap = std::max(bytes, size_t(16384));
    if ((e = hipHostMalloc(&t.host, cap, hipHostMallocDefault)) != hipSuccess) {
      (void)hipGetLastError();
      set_err(h, "hipHostMalloc of a descriptor staging buffer failed");
      return MUON_ERR_OUT_OF_MEMORY;
    }
    t.host_cap = cap;
  }
  std::memcpy(t.host, data, bytes);
  if ((e = hipMemcpyAsync(t.dev, t.host, bytes, hipMemcpyHostToDevice, stream)) != hipSuccess)
    return device_fail(h, "hipMemcpyAsync", e);
  if ((e = hipEventRecord(t.staged, stream)) != hipSuccess) return device_fail(h, "hipEventRecord", e);
  t.pending = true;
  t.last.assign(static_cast<const char*>(data), static_cast<const char*>(data) + bytes);
  return MUON_OK;
}

// Orders `stream` after the previous call's work when that ran on another
// stream (the workspace and the tables are shared by all calls).
muon_status_t begin_call(muon_handle_t h, hipStream_t stream) {
  if (h->have_last && stream != h->last_stream) {
    const hipError_t e = hipStreamWaitEvent(stream, h->call_done, 0);
    if (e != hipSuccess) return device_fail(h, "hipStreamWaitEvent", e);
  }
  return MUON_OK;
}

muon_status_t end_call(muon_handle_t h, hipStream_t stream) {
  const hipError_t e = hipEventRecord(h->call_done, stream);
  if (e != hipSuccess) return device_fail(h, "hipEventRecord", e);
  h->last_stream = stream;
  h->have_last = true;
  return MUON_OK;
}

bool create_table(DeviceTable& t) {
  return hipEventCreateWithFlags(&t.staged, hipEventDisableTiming) == hipSuccess;
}

void destroy_table(DeviceTable& t) {
  if (t.dev) (void)hipFree(t.dev);
  if (t.host) (void)hipHostFree(t.host);
  if (t.staged) (void)hipEventDestroy(t.staged);
  t = DeviceTable();
}

}  // namespace

// The last request of a handle in validated and planned form.  A training
// loop passes the same tensors, shapes and options every step, so the
// checks, the runtime queries about each buffer and the planning run once
// for them.  The key is the request's bytes: the entry array, the
// hyperparameters except lr and weight decay (they only change the
// descriptor table, rebuilt every call), the contents of every coefficient
// table, and the handle settings the plan depends on.
struct CallCache {
  bool valid = false;
  std::vector<char> key;
  std::vector<Item> items;
  CoeffTables tables;
  std::vector<Span> spans;
  Plan plan;
};

namespace {

CallCache* cache_of(muon_handle_t h) {
  if (!h->cache) h->cache = new (std::nothrow) CallCache();
  return h->cache;
}

void key_append(std::vector<char>& k, const void* p, size_t n) {
  const char* c = static_cast<const char*>(p);
  k.insert(k.end(), c, c + n);
}

// A coefficient table's contents, when its step count is one validation
// would accept (otherwise validation rejects the call anyway).
void key_coeffs(std::vector<char>& k, const float* c, int32_t steps) {
  if (c && steps > 0 && steps <= kMaxSteps) key_append(k, c, size_t(12) * size_t(steps));
}

void key_settings(std::vector<char>& k, const muon_handle* h) {
  key_append(k, &h->nstreams, sizeof h->nstreams);
  key_append(k, &h->grouping, sizeof h->grouping);
  key_append(k, &h->ws_limit, sizeof h->ws_limit);
}

bool step_key(std::vector<char>& k, const muon_param_t* params, int64_t n, const muon_hparams_t* hp,
              const muon_handle* h) {
  if (!hp || n < 0 || (n > 0 && !params)) return false;
  k.clear();
  k.reserve(size_t(n) * sizeof(muon_param_t) + 256);
  k.push_back('S');
  muon_hparams_t hc = *hp;
  hc.lr = 0.f;
  hc.weight_decay = 0.f;
  hc.ns_coeffs = nullptr;
  key_append(k, &hc, sizeof hc);
  key_coeffs(k, hp->ns_coeffs, hp->ns_steps);
  for (int64_t i = 0; i < n; ++i) {
    muon_param_t pc = params[i];
    pc.ns_coeffs = nullptr;
    key_append(k, &pc, sizeof pc);
    key_coeffs(k, params[i].ns_coeffs, params[i].ns_steps);
  }
  key_settings(k, h);
  return true;
}

bool orth_key(std::vector<char>& k, const void* const* in, void* const* out, const int64_t* rows,
              const int64_t* cols, int64_t n, int dtype, int32_t ns_steps, const float* coeffs, float eps,
              int prec, const muon_handle* h) {
  if (n < 0 || (n > 0 && (!in || !out || !rows || !cols))) return false;
  k.clear();
  k.push_back('O');
  key_append(k, &n, sizeof n);
  key_append(k, &dtype, sizeof dtype);
  key_append(k, &ns_steps, sizeof ns_steps);
  key_append(k, &eps, sizeof eps);
  key_append(k, &prec, sizeof prec);
  key_coeffs(k, coeffs, ns_steps);
  key_append(k, in, size_t(n) * sizeof(void*));
  key_append(k, out, size_t(n) * sizeof(void*));
  key_append(k, rows, size_t(n) * sizeof(int64_t));
  key_append(k, cols, size_t(n) * sizeof(int64_t));
  key_settings(k, h);
  return true;
}

MatDesc make_desc(const Item& it, double lr, double wd) {
  MatDesc d{};
  d.W = it.W; d.g = it.g; d.buf = it.buf; d.out = it.out;
  d.rows = int32_t(it.rows); d.cols = int32_t(it.cols);
  d.transposed = it.rows > it.cols ? 1 : 0;
  d.ld = it.ld; d.bstride = it.bs; d.ld_b = it.ld_b; d.bstride_b = it.bs_b;
  d.rb = int32_t(it.rb);
  const bool blocks = it.rb < it.rows;
  d.dense = (it.ld == it.cols && it.ld_b == it.cols && !blocks) ? 1 : 0;
  const auto al16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
  // 8 consecutive elements of g and buf at 16-byte aligned addresses: over
  // the flat index when dense, else within a row (every row start aligned)
  const bool rows8 = it.cols % 8 == 0 && it.ld % 8 == 0 && it.ld_b % 8 == 0 &&
                     (!blocks || (it.bs % 8 == 0 && it.bs_b % 8 == 0));
  d.vec_ok = (d.dense ? (it.rows * it.cols) % 8 == 0 : rows8) && al16(it.g) && (!it.buf || al16(it.buf)) ? 1 : 0;
  d.vec4_ok = (it.cols % 4 == 0 && it.ld % 4 == 0 && (!blocks || it.bs % 4 == 0)) && al16(it.W ? it.W : it.out) ? 1 : 0;
  d.row8_ok = rows8 && al16(it.g) && (!it.buf || al16(it.buf)) ? 1 : 0;
  double scale = 1.0;
  if (it.scale_mode == 0) scale = 0.2 * std::sqrt(double(std::max(it.rows, it.cols)));
  else if (it.scale_mode == 2) scale = std::sqrt(std::max(1.0, double(it.rows) / double(it.cols)));
  // the post-processing factor multiplies both terms of the update
  d.upd_scale = float(it.post_scale * lr * scale);
  d.decay = float(it.post_scale * (1.0 - lr * wd));
  return d;
}

muon_status_t execute(muon_handle_t h, const std::vector<Item>& items, const Plan& plan,
                      double lr, double wd, const StepScalars& sc, bool ns_f32,
                      const CoeffTables& tables, hipStream_t stream) {
  DeviceGuard dg(h->device);
  if (!dg.ok) { set_err(h, "cannot select device %d", h->device); return MUON_ERR_DEVICE; }
  // Units of work, in plan order: one chunk, or a group of chunks whose
  // products run as one launch per product and step (muon::run_group):
  // chunks whose Gram launch leaves CUs idle in its last round (occupancy
  // below 0.9), that can share the 256 x 256 kernel, with the same step
  // count and parameter dtype, at most kGroupMax to a group.  A group's
  // members each keep their own workspace region.  Groups are formed when
  // the call runs on one stream: with two, such chunks overlap on the two
  // streams instead, which measured faster (one block, hidden 2048: 2.17
  // against 2.36 ms per step; its two chunks' Gram products differ in K, and
  // a grouped round waits for the longest tile, where a chunk on its own
  // stream moves on to its next product).  On one stream, groups measured
  // 2.51 against 2.95 ms.
  const bool concurrent = h->nstreams > 1 && h->side != nullptr;
  int cus = 256;
  (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->device);
  auto geom_of = [&](const Chunk& c) {
    ChunkGeom g{};
    g.s = int32_t(c.s); g.l = int32_t(c.l); g.S = int32_t(c.S); g.L = int32_t(c.L);
    g.nmat = int32_t(c.count);
    g.ns_f32 = ns_f32 ? 1 : 0;
    g.grad_dtype = c.gdt == MUON_BF16 ? muon::DT_BF16 : muon::DT_F32;
    g.param_dtype = c.pdt == MUON_BF16 ? muon::DT_BF16 : muon::DT_F32;
    return g;
  };
  auto steps_of = [&](const Chunk& c) { return int(tables[size_t(c.cset)].size() / 3); };
  auto idle_of = [&](const Chunk& c) {
    const bool tile = !ns_f32 && c.S % 256 == 0;
    const int64_t t = tile ? c.S / 256 : c.S / 128;
    const int64_t tiles = t * (t + 1) / 2 * c.count, slots = int64_t(tile ? cus : 2 * cus);
    return double(tiles) / double(((tiles + slots - 1) / slots) * slots) < 0.9;
  };
  struct Unit {
    std::vector<size_t> members;  // chunk indices, plan order
    std::vector<size_t> off;      // each member's workspace offset inside the unit's region
    size_t bytes = 0;
    bool idle = false;
  };
  const size_t nch = plan.chunks.size();
  std::vector<Unit> units;
  std::vector<char> on_side;
  bool two = false;
  size_t slot = 0, need = 0;
  // (a second pass without groups when the groups' regions would pass the
  // workspace limit)
  for (int pass = 0; pass < 2; ++pass) {
  const bool allow_groups = h->grouping && !concurrent && pass == 0;
  units.clear();
  std::vector<char> grouped(nch, 0);
  if (allow_groups) {
    std::map<std::pair<int, int32_t>, size_t> open;  // (steps, param dtype) -> unit with room
    for (size_t ci = 0; ci < nch; ++ci) {
      const Chunk& c = plan.chunks[ci];
      if (!idle_of(c) || !muon::group_eligible(geom_of(c), steps_of(c))) continue;
      const std::pair<int, int32_t> key{steps_of(c), c.pdt};
      auto it = open.find(key);
      if (it == open.end() || units[it->second].members.size() >= size_t(muon::kGroupMax)) {
        units.emplace_back();
        open[key] = units.size() - 1;
        it = open.find(key);
      }
      units[it->second].members.push_back(ci);
      grouped[ci] = 1;
    }
    // a group of one is a plain chunk
    for (Unit& u : units)
      if (u.members.size() == 1) grouped[u.members[0]] = 0;
    units.erase(std::remove_if(units.begin(), units.end(), [](const Unit& u) { return u.members.size() < 2; }),
                units.end());
  }
  for (size_t ci = 0; ci < nch; ++ci)
    if (!grouped[ci]) {
      units.emplace_back();
      units.back().members.push_back(ci);
    }
  std::sort(units.begin(), units.end(), [](const Unit& a, const Unit& b) { return a.members[0] < b.members[0]; });
  for (Unit& u : units) {
    for (size_t ci : u.members) {
      u.off.push_back(u.bytes);
      u.bytes += align256(plan.chunks[ci].bytes);
    }
    u.idle = u.members.size() > 1 || idle_of(plan.chunks[u.members[0]]);
  }
  // Which units run on the second stream: idle ones alternate between the
  // streams, so one unit's idle CUs take the other's work; units that fill
  // every round stay on the caller's stream (two such kernels side by side
  // share the XCDs' L2 less well: measured slower).  The second slot of
  // workspace is used only when it fits under the workspace limit.
  on_side.assign(units.size(), 0);
  two = false;
  if (h->nstreams > 1 && h->side && units.size() > 1) {
    int low = 0;
    for (size_t ui = 0; ui < units.size(); ++ui) {
      if (units[ui].idle) on_side[ui] = (low++ % 2 == 0);
      two = two || on_side[ui];
    }
  }
  // each slot sized for the units that run on its stream
  size_t main_bytes = 0, side_bytes = 0;
  for (size_t ui = 0; ui < units.size(); ++ui)
    (on_side[ui] ? side_bytes : main_bytes) = std::max(on_side[ui] ? side_bytes : main_bytes, units[ui].bytes);
  slot = align256(main_bytes);
  if (two && h->ws_limit && slot + side_bytes > h->ws_limit) {
    two = false;
    std::fill(on_side.begin(), on_side.end(), 0);
  }
  if (!two && main_bytes < side_bytes) main_bytes = side_bytes;
  need = two ? slot + side_bytes : main_bytes;
  const bool any_group = std::any_of(units.begin(), units.end(), [](const Unit& u) { return u.members.size() > 1; });
  if (!(any_group && h->ws_limit && need > h->ws_limit)) break;
  }
  muon_status_t st = ensure_workspace(h, need);
  if (st != MUON_OK) return st;
  if (h->log) {
    std::fprintf(stderr, "muon: %zu matrices in %zu chunks (%zu units), %s NS, %s, workspace %zu bytes\n",
                 plan.order.size(), plan.chunks.size(), units.size(), ns_f32 ? "fp32" : "bf16",
                 two ? "two streams" : "one stream", h->ws_bytes);
    for (size_t ui = 0; ui < units.size(); ++ui)
      for (size_t mi = 0; mi < units[ui].members.size(); ++mi) {
        const size_t ci = units[ui].members[mi];
        const Chunk& c = plan.chunks[ci];
        std::fprintf(stderr,
                     "muon:   chunk %zu: %lld matrices of %lld x %lld (padded %lld x %lld), K = %zu, "
                     "coefficient set %d, X^T %s, %s stream, %zu workspace bytes%s\n",
                     ci, (long long)c.count, (long long)c.s, (long long)c.l, (long long)c.S, (long long)c.L,
                     tables[size_t(c.cset)].size() / 3, int(c.cset), c.keeps_xt ? "kept" : "not kept",
                     on_side[ui] ? "second" : "caller's", c.bytes,
                     units[ui].members.size() > 1 ? (mi == 0 ? ", grouped launches (first of the group)"
                                                            : ", grouped launches") : "");
      }
  }
  if ((st = begin_call(h, stream)) != MUON_OK) return st;
  // From here every exit records call_done, so that later calls wait for
  // whatever this one managed to enqueue.
  const auto fail = [&](muon_status_t s) { (void)end_call(h, stream); return s; };
  std::vector<MatDesc> table(plan.order.size());
  for (size_t p = 0; p < plan.order.size(); ++p) table[p] = make_desc(items[size_t(plan.order[p])], lr, wd);
  if ((st = upload_table(h, h->mats, table.data(), table.size() * sizeof(MatDesc), stream)) != MUON_OK)
    return fail(st);
  const MatDesc* d_desc = static_cast<const MatDesc*>(h->mats.dev);
  // The launches of the call on stream `s`: fork, every chunk, join.
  auto launch_all = [&](hipStream_t s) -> muon_status_t {
    if (two) {
      hipError_t e = hipEventRecord(h->fork, s);
      if (e == hipSuccess) e = hipStreamWaitEvent(h->side, h->fork, 0);
      if (e != hipSuccess) return device_fail(h, "fork", e);
    }
    hipError_t launch_err = hipSuccess;
    for (size_t ui = 0; ui < units.size() && launch_err == hipSuccess; ++ui) {
      const Unit& u = units[ui];
      const bool odd = on_side[ui] != 0;
      char* const base = static_cast<char*>(h->ws) + (odd ? slot : 0);
      const hipStream_t cs = odd ? h->side : s;
      muon::GroupMember gm[muon::kGroupMax];
      for (size_t mi = 0; mi < u.members.size(); ++mi) {
        const Chunk& c = plan.chunks[u.members[mi]];
        char* const ws = base + u.off[mi];
        ChunkBuffers b{};
        b.X[0] = ws + c.off_X[0]; b.X[1] = ws + c.off_X[1];
        b.XT[0] = c.keeps_xt ? ws + c.off_XT[0] : nullptr;
        b.XT[1] = c.keeps_xt ? ws + c.off_XT[1] : nullptr;
        b.A = ws + c.off_A; b.B = ws + c.off_B;
        b.partials = reinterpret_cast<double*>(ws + c.off_part);
        b.rscale = reinterpret_cast<double*>(ws + c.off_r);
        b.xscale = reinterpret_cast<float*>(b.rscale + c.count);
        b.sync = muon::chunk_is_small(c.s, c.l, ns_f32) ? reinterpret_cast<unsigned*>(ws + c.off_sync) : nullptr;
        gm[mi] = muon::GroupMember{geom_of(c), d_desc + c.first, b, tables[size_t(c.cset)].data()};
      }
      muon::LaunchTimer* const tmr = h->profiling ? &h->timer : nullptr;
      const int K = steps_of(plan.chunks[u.members[0]]);
      if (u.members.size() == 1)
        launch_err = muon::run_chunk(gm[0].geom, gm[0].desc, gm[0].wb, sc, gm[0].coeffs, K, cs, tmr);
      else
        launch_err = muon::run_group(gm, int(u.members.size()), sc, K, cs, tmr);
    }
    if (two) {  // joined even after a failed launch, so later calls stay ordered
      hipError_t e = hipEventRecord(h->join, h->side);
      if (e == hipSuccess) e = hipStreamWaitEvent(s, h->join, 0);
      if (e != hipSuccess) {
        (void)hipStreamSynchronize(h->side);  // not joined: wait on the host instead
        if (launch_err == hipSuccess) return device_fail(h, "join", e);
      }
    }
    if (launch_err != hipSuccess) return device_fail(h, "kernel launch", launch_err);
    return MUON_OK;
  };
  if ((st = launch_all(stream)) != MUON_OK) return fail(st);
  return end_call(h, stream);
}

// AdamW: checks, then one launch per (param, grad) dtype pair over the
// tensors of that pair.
muon_status_t validate_adamw(const muon_adamw_param_t* params, int64_t n, const muon_adamw_hparams_t* hp,
                             Msg& msg, std::vector<Span>* spans = nullptr) {
  if (!hp) { msg.set("hparams is NULL"); return MUON_ERR_INVALID_ARGUMENT; }
  if (!std::isfinite(hp->lr) || !std::isfinite(hp->weight_decay) || !std::isfinite(hp->eps) ||
      !(hp->eps > 0.f)) {
    msg.set("lr and weight_decay must be finite, eps finite and > 0");
    return MUON_ERR_INVALID_ARGUMENT;
  }
  if (!(hp->beta1 >= 0.f && hp->beta1 < 1.f) || !(hp->beta2 >= 0.f && hp->beta2 < 1.f)) {
    msg.set("beta1 and beta2 must be in [0, 1)");
    return MUON_ERR_INVALID_ARGUMENT;
  }
  if (hp->step < 1) { msg.set("step must be >= 1"); return MUON_ERR_INVALID_ARGUMENT; }
  if (hp->reserved != 0) { msg.set("reserved must be 0"); return MUON_ERR_INVALID_ARGUMENT; }
  if (n < 0) { msg.set("n must be >= 0"); return MUON_ERR_INVALID_ARGUMENT; }
  if (n > 0 && !params) { msg.set("params is NULL"); return MUON_ERR_INVALID_ARGUMENT; }
  std::vector<Run> runs;
  for (int64_t i = 0; i < n; ++i) {
    const muon_adamw_param_t& p = params[i];
    if (p.numel < 0 || p.numel > (int64_t(1) << 40)) { msg.set("entry %lld: numel out of range", (long long)i); return MUON_ERR_INVALID_ARGUMENT; }
    if (p.numel == 0) continue;
    if (!p.param || !p.grad || !p.exp_avg || !p.exp_avg_sq) { msg.set("entry %lld: NULL pointer", (long long)i); return MUON_ERR_INVALID_ARGUMENT; }
    if (!dtype_ok(p.param_dtype) || !dtype_ok(p.grad_dtype)) { msg.set("entry %lld: unknown dtype", (long long)i); return MUON_ERR_INVALID_ARGUMENT; }
    const uintptr_t P = reinterpret_cast<uintptr_t>(p.param), G = reinterpret_cast<uintptr_t>(p.grad),
                    M = reinterpret_cast<uintptr_t>(p.exp_avg), V = reinterpret_cast<uintptr_t>(p.exp_avg_sq);
    const size_t ps = dtype_size(p.param_dtype), gs = dtype_size(p.grad_dtype);
    if (P % ps || G % gs || M % 4 || V % 4) { msg.set("entry %lld: pointer not aligned to its element size", (long long)i); return MUON_ERR_INVALID_ARGUMENT; }
    const uintptr_t ne = uintptr_t(p.numel);
    runs.push_back({P, ne * ps, ne * ps, 1, true});
    runs.push_back({G, ne * gs, ne * gs, 1, false});
    runs.push_back({M, ne * 4, ne * 4, 1, true});
    runs.push_back({V, ne * 4, ne * 4, 1, true});
    if (spans)
      for (const Span& sp : {Span{P, P + ne * ps}, Span{G, G + ne * gs}, Span{M, M + ne * 4}, Span{V, V + ne * 4}})
        spans->push_back(sp);
  }
  if (!runs_disjoint(runs)) { msg.set("param, grad and moment buffers overlap"); return MUON_ERR_INVALID_ARGUMENT; }
  return MUON_OK;
}

// Launching calls only (host-only validation takes any address): every
// buffer must start in device memory of the handle's device (or managed
// memory), and if it reaches beyond the allocation that holds its start, its
// last byte must be such memory too (a tensor may span several allocations
// mapped back to back).  A host pointer, another device's memory, or a view
// that runs past its allocation into unmapped addresses is an error here
// instead of a fault in a kernel.
muon_status_t check_device_spans(muon_handle_t h, const Span* spans, size_t n) {
  const auto device_mem = [&](uintptr_t addr) {
    hipPointerAttribute_t a{};
    if (hipPointerGetAttributes(&a, reinterpret_cast<const void*>(addr)) != hipSuccess) {
      (void)hipGetLastError();
      return false;
    }
    return a.isManaged || a.type == hipMemoryTypeManaged || (a.type == hipMemoryTypeDevice && a.device == h->device);
  };
  for (size_t i = 0; i < n; ++i) {
    const Span& s = spans[i];
    if (s.hi <= s.lo) continue;
    if (!device_mem(s.lo)) {
      set_err(h, "buffer at %p is not device memory of device %d", reinterpret_cast<void*>(s.lo), h->device);
      return MUON_ERR_INVALID_ARGUMENT;
    }
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, reinterpret_cast<hipDeviceptr_t>(s.lo)) == hipSuccess && base &&
        s.hi <= reinterpret_cast<uintptr_t>(base) + size)
      continue;
    (void)hipGetLastError();
    if (!device_mem(s.hi - 1)) {
      set_err(h, "buffer at %p reaches past the end of its allocation: its last byte (%p) is not device memory of device %d",
              reinterpret_cast<void*>(s.lo), reinterpret_cast<void*>(s.hi - 1), h->device);
      return MUON_ERR_INVALID_ARGUMENT;
    }
  }
  return MUON_OK;
}

muon_status_t check_device_spans(muon_handle_t h, const std::vector<Span>& spans) {
  return check_device_spans(h, spans.data(), spans.size());
}

std::vector<float> coefficient_table(int K, const float* coeffs) {
  std::vector<float> t(size_t(3) * size_t(K));
  for (int k = 0; k < K; ++k)
    for (int j = 0; j < 3; ++j) t[size_t(3 * k + j)] = coeffs ? coeffs[3 * k + j] : kLegacyQuintic[j];
  return t;
}

std::vector<int> step_counts(const CoeffTables& tables) {
  std::vector<int> k;
  for (const auto& t : tables) k.push_back(int(t.size() / 3));
  return k;
}

// ---------------------------------------------------------------------------
// Allocation-free orthogonalisation (ns_orthogonalize_batched_noalloc).
// Its workspace and descriptor table live in `scratch`, a fixed array of this
// library in device memory: each device the library runs on holds its own
// copy until the process ends.  In host code `scratch` names a host-side
// stand-in, never the device memory: its device address on each device is
// taken once with hipGetSymbolAddress (muon_create, with the device current)
// and kept per device; only that address reaches kernels.  Every call on a
// device shares that device's array, so calls that overlap in time on one
// device race (one at a time per device, or ordered on one stream).
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = size_t(64) << 20;
constexpr int kNoAllocMaxMats = 64;
constexpr size_t kScratchDescBytes = (kNoAllocMaxMats * sizeof(MatDesc) + 255) & ~size_t(255);
constexpr int kMaxDevices = 64;

}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

// This device's address of `scratch` (device current), resolved once per
// device; null when the runtime cannot give it.
void* resolve_scratch(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch_addr[device] = p;
  }
  return g_scratch_addr[device];
}

// Do [a, a + na) and [b, b + nb) share a byte?
bool bytes_meet(uintptr_t a, uintptr_t na, uintptr_t b, uintptr_t nb) { return a < b + nb && b < a + na; }

}  // namespace

extern "C" {

int muon_abi_version(void) { return MUON_HIP_ABI_VERSION; }

const char* muon_status_string(muon_status_t s) {
  switch (s) {
    case MUON_OK: return "MUON_OK";
    case MUON_ERR_INVALID_ARGUMENT: return "MUON_ERR_INVALID_ARGUMENT";
    case MUON_ERR_UNSUPPORTED: return "MUON_ERR_UNSUPPORTED";
    case MUON_ERR_OUT_OF_MEMORY: return "MUON_ERR_OUT_OF_MEMORY";
    case MUON_ERR_DEVICE: return "MUON_ERR_DEVICE";
  }
  return "MUON_ERR_UNKNOWN";
}

const char* muon_last_error(muon_handle_t h) { return h ? h->err : "NULL handle"; }

muon_status_t muon_create(muon_handle_t* out, int device) {
  if (!out) return MUON_ERR_INVALID_ARGUMENT;
  *out = nullptr;
  int count = 0;
  if (hipGetDeviceCount(&count) != hipSuccess || count <= 0) { (void)hipGetLastError(); return MUON_ERR_DEVICE; }
  if (device < 0 || device >= count) return MUON_ERR_INVALID_ARGUMENT;
  muon_handle* h = new (std::nothrow) muon_handle();
  if (!h) return MUON_ERR_OUT_OF_MEMORY;
  h->device = device;
  const char* lg = std::getenv("MUON_HIP_LOG");
  h->log = lg && *lg && std::strcmp(lg, "0") != 0;

  DeviceGuard dg(device);
  auto drop_side = [h]() {
    if (h->side) (void)hipStreamDestroy(h->side);
    if (h->fork) (void)hipEventDestroy(h->fork);
    if (h->join) (void)hipEventDestroy(h->join);
    h->side = nullptr; h->fork = h->join = nullptr;
    h->nstreams = 1;
  };
  // the second stream has the default priority, like every stream here
  if (dg.ok &&
      (hipStreamCreateWithFlags(&h->side, hipStreamNonBlocking) != hipSuccess ||
       hipEventCreateWithFlags(&h->fork, hipEventDisableTiming) != hipSuccess ||
       hipEventCreateWithFlags(&h->join, hipEventDisableTiming) != hipSuccess)) {
    (void)hipGetLastError();
    drop_side();  // run on the caller's stream alone
  }
  if (!dg.ok || !create_table(h->mats) || !create_table(h->adams) ||
      hipEventCreateWithFlags(&h->call_done, hipEventDisableTiming) != hipSuccess) {
    destroy_table(h->mats);
    destroy_table(h->adams);
    if (h->call_done) (void)hipEventDestroy(h->call_done);
    drop_side();
    delete h;
    return MUON_ERR_DEVICE;
  }
  // the allocation-free entry point's array on this device (once per device)
  h->scratch = resolve_scratch(device);

  *out = h;
  return MUON_OK;
}

muon_status_t muon_destroy(muon_handle_t h) {
  if (!h) return MUON_ERR_INVALID_ARGUMENT;
  muon_status_t st = MUON_OK;
  {
    DeviceGuard dg(h->device);
    if (wait_idle(h) != MUON_OK) st = MUON_ERR_DEVICE;
    for (DeviceTable* t : {&h->mats, &h->adams})  // staging copies still in flight
      if (t->pending && hipEventSynchronize(t->staged) != hipSuccess) st = MUON_ERR_DEVICE;
    if (h->ws) (void)hipFree(h->ws);
    destroy_table(h->mats);
    destroy_table(h->adams);
    if (h->call_done) (void)hipEventDestroy(h->call_done);
    if (h->side) (void)hipStreamDestroy(h->side);
    if (h->fork) (void)hipEventDestroy(h->fork);
    if (h->join) (void)hipEventDestroy(h->join);
    delete h->cache;
    h->timer.destroy();
  }
  delete h;
  return st;
}

muon_status_t muon_set_streams(muon_handle_t h, int streams) {
  if (!h || (streams != 1 && streams != 2)) return MUON_ERR_INVALID_ARGUMENT;
  if (streams == 2 && !h->side) {
    set_err(h, "the second stream could not be created");
    return MUON_ERR_DEVICE;
  }
  h->nstreams = streams;
  return MUON_OK;
}

muon_status_t muon_set_grouping(muon_handle_t h, int enable) {
  if (!h || (enable != 0 && enable != 1)) return MUON_ERR_INVALID_ARGUMENT;
  h->grouping = enable;
  return MUON_OK;
}

muon_status_t muon_reserve(muon_handle_t h, size_t bytes) {
  if (!h) return MUON_ERR_INVALID_ARGUMENT;
  DeviceGuard dg(h->device);
  if (!dg.ok) return MUON_ERR_DEVICE;
  return ensure_workspace(h, bytes);
}

muon_status_t muon_set_workspace_limit(muon_handle_t h, size_t bytes) {
  if (!h) return MUON_ERR_INVALID_ARGUMENT;
  h->ws_limit = bytes;
  return MUON_OK;
}

size_t muon_workspace_bytes(muon_handle_t h) { return h ? h->ws_bytes : 0; }

muon_status_t muon_profile_enable(muon_handle_t h, int enable) {
  if (!h) return MUON_ERR_INVALID_ARGUMENT;
  h->profiling = enable != 0;
  return MUON_OK;
}

muon_status_t muon_profile_read(muon_handle_t h, muon_kernel_stats_t* out, int cap, int* n,
                                int reset) {
  static const char* const kNames[muon::KK_COUNT] = {
      "momentum_norm", "norm_finalize", "rescale", "gram_syrk",
      "poly_syrk", "update_gemm", "update_apply_gemm", "apply_x0", "adamw", "ns_small"};
  if (!h || (cap > 0 && !out)) return MUON_ERR_INVALID_ARGUMENT;
  DeviceGuard dg(h->device);
  const bool ok = h->timer.collect();
  if (n) *n = muon::KK_COUNT;
  for (int k = 0; k < cap && k < muon::KK_COUNT; ++k) {
    const EventTimer::Acc& a = h->timer.acc[k];
    out[k].name = kNames[k];
    out[k].launches = a.launches;
    out[k].total_ms = a.ms;
    out[k].flops = a.flops;
    out[k].exec_flops = a.exec;
    out[k].bytes = a.bytes;
  }
  if (reset) h->timer.reset();
  if (!ok) { set_err(h, "event timing failed"); return MUON_ERR_DEVICE; }
  return MUON_OK;
}

muon_status_t muon_validate_step(const muon_param_t* params, int64_t n, const muon_hparams_t* hp,
                                 char* msg, size_t msg_len) {
  Msg m{msg, msg_len};
  if (msg && msg_len) msg[0] = '\0';
  return validate_step(params, n, hp, nullptr, nullptr, m);
}

muon_status_t muon_plan_step(const muon_param_t* params, int64_t n, const muon_hparams_t* hp,
                             muon_chunk_info_t* chunks, int64_t cap, int64_t* n_chunks,
                             size_t* workspace_bytes, int64_t* order) {
  Msg m{nullptr, 0};
  std::vector<Item> items;
  CoeffTables tables;
  muon_status_t st = validate_step(params, n, hp, &items, &tables, m);
  if (st != MUON_OK) return st;
  if (cap > 0 && !chunks) return MUON_ERR_INVALID_ARGUMENT;
  const Plan plan = make_plan(items, hp->max_chunk_elems, hp->ns_precision == MUON_NS_F32, step_counts(tables));
  if (n_chunks) *n_chunks = int64_t(plan.chunks.size());
  if (workspace_bytes) *workspace_bytes = plan.ws_bytes;
  for (int64_t i = 0; i < cap && i < int64_t(plan.chunks.size()); ++i) {
    const Chunk& c = plan.chunks[size_t(i)];
    muon_chunk_info_t& o = chunks[i];
    o.s = c.s; o.l = c.l; o.s_pad = c.S; o.l_pad = c.L;
    o.first = c.first; o.count = c.count;
    o.param_dtype = c.pdt; o.grad_dtype = c.gdt;
    o.ns_steps = int32_t(tables[size_t(c.cset)].size() / 3);
    o.coeff_set = c.cset;
    o.workspace_bytes = c.bytes;
  }
  if (order)
    for (size_t p = 0; p < plan.order.size(); ++p) order[p] = items[size_t(plan.order[p])].flat;
  return MUON_OK;
}

muon_status_t muon_step(muon_handle_t h, const muon_param_t* params, int64_t n,
                        const muon_hparams_t* hp, void* stream) {
  if (!h) return MUON_ERR_INVALID_ARGUMENT;
  h->err[0] = '\0';
  char buf[256] = {0};
  Msg m{buf, sizeof buf};
  CallCache local;
  CallCache* c = cache_of(h);
  std::vector<char> key;
  const bool keyed = c && step_key(key, params, n, hp, h);
  if (!c) c = &local;
  muon_status_t st = MUON_OK;
  const bool hit = keyed && c->valid && c->key == key;
  if (hit) {
    // the same request as the last one: only lr and weight decay may differ
    if (!std::isfinite(hp->lr) || !std::isfinite(hp->weight_decay)) {
      set_err(h, "lr, beta, weight_decay must be finite and eps finite and >= 0");
      return MUON_ERR_INVALID_ARGUMENT;
    }
  } else {
    c->valid = false;
    c->items.clear();
    c->spans.clear();
    st = validate_step(params, n, hp, &c->items, &c->tables, m, &c->spans);
    if (st != MUON_OK) { set_err(h, "%s", buf); return st; }
    c->plan = make_plan(c->items, hp->max_chunk_elems, hp->ns_precision == MUON_NS_F32, step_counts(c->tables));
    c->valid = keyed;
    if (keyed) c->key.swap(key);
  }
  const std::vector<Item>& items = c->items;
  const CoeffTables& tables = c->tables;
  const Plan& plan = c->plan;
  if (items.empty()) return MUON_OK;
  // the runtime's view of the buffers was checked when this request first came
  if (!hit && (st = check_device_spans(h, c->spans)) != MUON_OK) {
    c->valid = false;
    return st;
  }
  const bool f32 = hp->ns_precision == MUON_NS_F32;
  StepScalars sc{};
  sc.beta = hp->beta;
  sc.one_minus_beta = 1.0f - hp->beta;
  sc.nesterov = hp->nesterov;
  sc.momentum = 1;
  sc.eps = hp->eps;
  sc.final_kind = 0;
  return execute(h, items, plan, hp->lr, hp->weight_decay, sc, f32, tables,
                 static_cast<hipStream_t>(stream));
}

muon_status_t muon_adamw_step(muon_handle_t h, const muon_adamw_param_t* params, int64_t n,
                              const muon_adamw_hparams_t* hp, void* stream_) {
  if (!h) return MUON_ERR_INVALID_ARGUMENT;
  h->err[0] = '\0';
  char buf[256] = {0};
  Msg m{buf, sizeof buf};
  std::vector<Span> spans;
  muon_status_t st = validate_adamw(params, n, hp, m, &spans);
  if (st != MUON_OK) { set_err(h, "%s", buf); return st; }
  if ((st = check_device_spans(h, spans)) != MUON_OK) return st;
  const hipStream_t stream = static_cast<hipStream_t>(stream_);
  // tensors grouped by dtype pair; workgroup ranges per group
  std::vector<muon::AdamDesc> table;
  struct Group { int pdt, gdt; size_t first, count; int64_t blocks; double bytes; };
  std::vector<Group> groups;
  for (int pdt : {MUON_BF16, MUON_F32})
    for (int gdt : {MUON_BF16, MUON_F32}) {
      Group gr{pdt, gdt, table.size(), 0, 0, 0.0};
      for (int64_t i = 0; i < n; ++i) {
        const muon_adamw_param_t& p = params[i];
        if (p.numel == 0 || p.param_dtype != pdt || p.grad_dtype != gdt) continue;
        muon::AdamDesc d{};
        d.p = p.param; d.g = p.grad; d.m = p.exp_avg; d.v = p.exp_avg_sq;
        d.numel = p.numel;
        d.first_block = gr.blocks;
        const auto al16 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; };
        d.vec_ok = p.numel % 8 == 0 && al16(p.param) && al16(p.grad) && al16(p.exp_avg) && al16(p.exp_avg_sq);
        gr.blocks += (p.numel + muon::kAdamElemsPerBlock - 1) / muon::kAdamElemsPerBlock;
        gr.bytes += double(p.numel) * (2.0 * dtype_size(pdt) + dtype_size(gdt) + 16.0);
        table.push_back(d);
        ++gr.count;
      }
      if (gr.count) groups.push_back(gr);
    }
  if (table.empty()) return MUON_OK;
  for (const Group& gr : groups)
    if (gr.blocks > int64_t(INT32_MAX)) { set_err(h, "too many elements in one dtype group"); return MUON_ERR_UNSUPPORTED; }
  DeviceGuard dg(h->device);
  if (!dg.ok) { set_err(h, "cannot select device %d", h->device); return MUON_ERR_DEVICE; }
  if ((st = begin_call(h, stream)) != MUON_OK) return st;
  // every exit from here records call_done (see execute)
  const auto fail = [&](muon_status_t s) { (void)end_call(h, stream); return s; };
  if ((st = upload_table(h, h->adams, table.data(), table.size() * sizeof(muon::AdamDesc), stream)) != MUON_OK)
    return fail(st);
  // scalars: bias corrections in double, then fp32
  const double t = double(hp->step);
  const double bc1 = 1.0 - std::pow(double(hp->beta1), t), bc2 = 1.0 - std::pow(double(hp->beta2), t);
  muon::AdamScalars sc{};
  sc.decay = float(1.0 - double(hp->lr) * double(hp->weight_decay));
  sc.beta1 = hp->beta1; sc.one_minus_beta1 = float(1.0 - double(hp->beta1));
  sc.beta2 = hp->beta2; sc.one_minus_beta2 = float(1.0 - double(hp->beta2));
  sc.step_size = float(double(hp->lr) / bc1);
  sc.inv_sqrt_bc2 = float(1.0 / std::sqrt(bc2));
  sc.eps = hp->eps;
  const muon::AdamDesc* d = static_cast<const muon::AdamDesc*>(h->adams.dev);
  for (const Group& gr : groups) {
    const hipError_t e = muon::run_adamw(d + gr.first, int(gr.count), gr.blocks,
                                         gr.pdt == MUON_BF16 ? muon::DT_BF16 : muon::DT_F32,
                                         gr.gdt == MUON_BF16 ? muon::DT_BF16 : muon::DT_F32, sc, gr.bytes,
                                         stream, h->profiling ? &h->timer : nullptr);
    if (e != hipSuccess) return fail(device_fail(h, "kernel launch", e));
  }
  return end_call(h, stream);
}

muon_status_t ns_orthogonalize_batched(muon_handle_t h, const void* const* in, void* const* out,
                                       const int64_t* rows, const int64_t* cols, int64_t n,
                                       muon_dtype_t dtype, int32_t ns_steps, const float* ns_coeffs,
                                       float eps, muon_ns_precision_t prec, void* stream) {
  if (!h) return MUON_ERR_INVALID_ARGUMENT;
  h->err[0] = '\0';
  char buf[256] = {0};
  Msg m{buf, sizeof buf};
  CallCache local;
  CallCache* c = cache_of(h);
  std::vector<char> key;
  const bool keyed = c && orth_key(key, in, out, rows, cols, n, dtype, ns_steps, ns_coeffs, eps, prec, h);
  if (!c) c = &local;
  muon_status_t st = MUON_OK;
  const bool f32 = prec == MUON_NS_F32;
  const bool hit = keyed && c->valid && c->key == key;
  if (!hit) {
    c->valid = false;
    c->items.clear();
    c->spans.clear();
    st = validate_orth(in, out, rows, cols, n, dtype, ns_steps, ns_coeffs, eps, prec, &c->items, m, &c->spans);
    if (st != MUON_OK) { set_err(h, "%s", buf); return st; }
    c->tables = CoeffTables{coefficient_table(ns_steps, ns_coeffs)};
    c->plan = make_plan(c->items, 0, f32, step_counts(c->tables));
    c->valid = keyed;
    if (keyed) c->key.swap(key);
  }
  const std::vector<Item>& items = c->items;
  const CoeffTables& tables = c->tables;
  const Plan& plan = c->plan;
  if (items.empty()) return MUON_OK;
  if (!hit && (st = check_device_spans(h, c->spans)) != MUON_OK) {
    c->valid = false;
    return st;
  }
  StepScalars sc{};
  sc.momentum = 0;
  sc.eps = eps;
  sc.final_kind = 1;
  return execute(h, items, plan, 0.0, 0.0, sc, f32, tables, static_cast<hipStream_t>(stream));
}


muon_status_t ns_orthogonalize_batched_noalloc(muon_handle_t h, const void* const* in, void* const* out,
                                               const int64_t* rows, const int64_t* cols, int64_t n,
                                               muon_dtype_t dtype, int32_t ns_steps, const float* ns_coeffs,
                                               float eps, muon_ns_precision_t prec, void* stream_) {
  if (!h) return MUON_ERR_INVALID_ARGUMENT;
  h->err[0] = '\0';
  char buf[256] = {0};
  Msg m{buf, sizeof buf};
  muon_status_t st = check_orth_args(in, out, rows, cols, n, dtype, ns_steps, ns_coeffs, eps, prec, m);
  if (st != MUON_OK) { set_err(h, "%s", buf); return st; }
  if (n > kNoAllocMaxMats) {
    set_err(h, "%lld matrices: the allocation-free entry point takes at most %d per call", (long long)n,
            kNoAllocMaxMats);
    return MUON_ERR_UNSUPPORTED;
  }
  if (n == 0) return MUON_OK;
  // the matrices, and the bytes each reads (when not in place) and writes
  const size_t es = dtype_size(dtype);
  Item items[kNoAllocMaxMats];
  Span spans[2 * kNoAllocMaxMats];
  size_t nspans = 0;
  for (int64_t i = 0; i < n; ++i) {
    if ((st = check_orth_matrix(in[i], out[i], rows[i], cols[i], es, i, m)) != MUON_OK) {
      set_err(h, "%s", buf);
      return st;
    }
    items[i] = orth_item(in[i], out[i], rows[i], cols[i], dtype, i);
    const uintptr_t a = reinterpret_cast<uintptr_t>(in[i]), b = reinterpret_cast<uintptr_t>(out[i]);
    const uintptr_t bytes = uintptr_t(rows[i]) * uintptr_t(cols[i]) * es;
    spans[nspans++] = {b, b + bytes};
    if (a != b) spans[nspans++] = {a, a + bytes};
  }
  // an output meets no other output and no input but its own exact in-place one
  for (int64_t i = 0; i < n; ++i) {
    const uintptr_t bi = reinterpret_cast<uintptr_t>(out[i]), ni = uintptr_t(rows[i] * cols[i]) * es;
    for (int64_t j = 0; j < n; ++j) {
      const uintptr_t aj = reinterpret_cast<uintptr_t>(in[j]), bj = reinterpret_cast<uintptr_t>(out[j]);
      const uintptr_t nj = uintptr_t(rows[j] * cols[j]) * es;
      if ((j != i && bytes_meet(bi, ni, bj, nj)) || (aj != bj && bytes_meet(bi, ni, aj, nj))) {
        set_err(h, "an output overlaps another buffer");
        return MUON_ERR_INVALID_ARGUMENT;
      }
    }
  }
  if (!h->scratch) {
    set_err(h, "the scratch array of device %d is not available", h->device);
    return MUON_ERR_DEVICE;
  }
  if ((st = check_device_spans(h, spans, nspans)) != MUON_OK) return st;
  // Plan, as make_plan does: buckets by (short side, long side) in order of
  // first appearance, sorted by work (stable), chunks of at most 2^29
  // elements, and here also no larger than the scratch array holds.
  const bool f32 = prec == MUON_NS_F32;
  const int K = ns_steps;
  int64_t bs[kNoAllocMaxMats], bl[kNoAllocMaxMats];
  int nb = 0;
  int bucket_of[kNoAllocMaxMats];
  for (int64_t i = 0; i < n; ++i) {
    const int64_t s = std::min(rows[i], cols[i]), l = std::max(rows[i], cols[i]);
    int b = 0;
    while (b < nb && !(bs[b] == s && bl[b] == l)) ++b;
    if (b == nb) { bs[nb] = s; bl[nb] = l; ++nb; }
    bucket_of[i] = b;
  }
  int korder[kNoAllocMaxMats];
  for (int b = 0; b < nb; ++b) korder[b] = b;
  const auto work = [&](int b) { return double(bs[b]) * double(bs[b]) * double(bl[b]) * std::max(1, K); };
  for (int x = 1; x < nb; ++x)  // stable insertion sort, largest work first
    for (int y = x; y > 0 && work(korder[y]) > work(korder[y - 1]); --y) std::swap(korder[y], korder[y - 1]);
  Chunk chunks[kNoAllocMaxMats];
  int64_t order[kNoAllocMaxMats];
  int nc = 0, np = 0;
  const size_t room = kScratchBytes - kScratchDescBytes;
  for (int kb = 0; kb < nb; ++kb) {
    const int b = korder[kb];
    int64_t members[kNoAllocMaxMats];
    int64_t nm = 0;
    for (int64_t i = 0; i < n; ++i)
      if (bucket_of[i] == b) members[nm++] = i;
    Chunk c{};
    c.s = bs[b]; c.l = bl[b];
    c.S = muon::round_up(c.s, muon::kPad);
    c.L = muon::round_up(c.l, muon::kPad);
    c.pdt = dtype; c.gdt = dtype; c.cset = 0;
    int64_t per = std::max<int64_t>(1, std::min<int64_t>(kMaxChunkMats, kDefaultChunkElems / (c.s * c.l)));
    per = std::min(per, nm);
    for (;; --per) {
      c.count = per;
      layout_chunk(c, f32, K);
      if (c.bytes <= room) break;
      if (per == 1) {
        set_err(h, "a %lld x %lld matrix needs %zu workspace bytes; the allocation-free entry point has %zu",
                (long long)c.s, (long long)c.l, c.bytes, room);
        return MUON_ERR_UNSUPPORTED;
      }
    }
    for (int64_t f = 0; f < nm; f += per) {
      Chunk cc = c;
      cc.first = np;
      cc.count = std::min(per, nm - f);
      layout_chunk(cc, f32, K);
      for (int64_t j = 0; j < cc.count; ++j) order[np++] = members[f + j];
      chunks[nc++] = cc;
    }
  }
  float ct[3 * kMaxSteps];
  for (int k = 0; k < K; ++k)
    for (int j = 0; j < 3; ++j) ct[3 * k + j] = ns_coeffs ? ns_coeffs[3 * k + j] : kLegacyQuintic[j];
  MatDesc table[kNoAllocMaxMats];
  for (int p = 0; p < np; ++p) table[p] = make_desc(items[order[p]], 0.0, 0.0);
  DeviceGuard dg(h->device);
  if (!dg.ok) { set_err(h, "cannot select device %d", h->device); return MUON_ERR_DEVICE; }
  const hipStream_t stream = static_cast<hipStream_t>(stream_);
  char* const base = static_cast<char*>(h->scratch);
  MatDesc* const d_desc = reinterpret_cast<MatDesc*>(base);
  char* const ws = base + kScratchDescBytes;
  hipError_t e = muon::put_descriptors(table, np, d_desc, stream);
  if (e != hipSuccess) return device_fail(h, "descriptor upload", e);
  StepScalars sc{};
  sc.momentum = 0;
  sc.eps = eps;
  sc.final_kind = 1;
  for (int ci = 0; ci < nc; ++ci) {
    const Chunk& c = chunks[ci];
    ChunkGeom g{};
    g.s = int32_t(c.s); g.l = int32_t(c.l); g.S = int32_t(c.S); g.L = int32_t(c.L);
    g.nmat = int32_t(c.count);
    g.ns_f32 = f32 ? 1 : 0;
    g.grad_dtype = g.param_dtype = dtype == MUON_BF16 ? muon::DT_BF16 : muon::DT_F32;
    ChunkBuffers b{};
    b.X[0] = ws + c.off_X[0]; b.X[1] = ws + c.off_X[1];
    b.XT[0] = c.keeps_xt ? ws + c.off_XT[0] : nullptr;
    b.XT[1] = c.keeps_xt ? ws + c.off_XT[1] : nullptr;
    b.A = ws + c.off_A; b.B = ws + c.off_B;
    b.partials = reinterpret_cast<double*>(ws + c.off_part);
    b.rscale = reinterpret_cast<double*>(ws + c.off_r);
    b.xscale = reinterpret_cast<float*>(b.rscale + c.count);
    b.sync = muon::chunk_is_small(c.s, c.l, f32) ? reinterpret_cast<unsigned*>(ws + c.off_sync) : nullptr;
    if ((e = muon::run_chunk(g, d_desc + c.first, b, sc, ct, K, stream, nullptr)) != hipSuccess)
      return device_fail(h, "kernel launch", e);
  }
  return MUON_OK;
}


muon_status_t muon_stream_copy(muon_handle_t h, void* dst, const void* src, size_t bytes, void* stream) {
  if (!h) return MUON_ERR_INVALID_ARGUMENT;
  h->err[0] = '\0';
  if (bytes == 0) return MUON_OK;
  const uintptr_t d = reinterpret_cast<uintptr_t>(dst), s = reinterpret_cast<uintptr_t>(src);
  if (!dst || !src || d % 16 || s % 16) {
    set_err(h, "dst and src must be non-NULL and 16-byte aligned");
    return MUON_ERR_INVALID_ARGUMENT;
  }
  if (bytes_meet(d, bytes, s, bytes)) {
    set_err(h, "dst and src overlap");
    return MUON_ERR_INVALID_ARGUMENT;
  }
  const Span spans[2] = {{d, d + bytes}, {s, s + bytes}};
  muon_status_t st = check_device_spans(h, spans, 2);
  if (st != MUON_OK) return st;
  DeviceGuard dg(h->device);
  if (!dg.ok) { set_err(h, "cannot select device %d", h->device); return MUON_ERR_DEVICE; }
  const hipError_t e = muon::stream_copy(dst, src, bytes, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MUON_OK : device_fail(h, "kernel launch", e);
}

}  // extern "C"
