// C ABI entry points: volume matrix, transform, batched transform, plan
// statistics, workspace control and kernel timing.  Plans are cached per
// (device, element size, layouts, ops, relabeling, workspace cap).
#include <algorithm>
#include <chrono>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <new>
#include <string>

#include "plan.hpp"

namespace costa {
namespace {

// Rectangles are cut at 4M elements: the kernels index a rectangle's
// elements in 32 bits and compute row and column from a float estimate of
// the quotient, exact up to one correction step below 2^24 units.
constexpr int64_t kMaxPieceElems = 1 << 22;

int elem_size(costa_dtype d) {
  switch (d) {
    case COSTA_R64: return 8;
    case COSTA_C128: return 16;
    case COSTA_R32: return 4;
    case COSTA_C64: return 8;
    default: return 0;  // not an element type
  }
}
bool is_complex(costa_dtype d) { return d == COSTA_C128 || d == COSTA_C64; }

#define HIP_OR_FAIL(expr)                                                                      \
  do {                                                                                         \
    hipError_t e_ = (expr);                                                                    \
    if (e_ != hipSuccess)                                                                      \
      return fail(COSTA_ERROR_DEVICE, std::string(#expr) + ": " + hipGetErrorString(e_));      \
  } while (0)

struct DevicePlan {
  HostPlan host;
  int device = -1;
  Piece* d_pieces = nullptr;
  int32_t* d_tasks = nullptr;
  int32_t* d_wide = nullptr;
  // per-call table: buffer pointers then pair parameters
  void* d_table = nullptr;
  void* h_staging = nullptr;  // pinned
  size_t table_bytes = 0;
  size_t nbufs = 0;
  std::vector<unsigned char> last_table;
  hipEvent_t table_event = nullptr;  // the last table upload (h_staging reusable after it)
  bool table_pending = false;
  hipEvent_t last_use = nullptr;     // end of the last call's launches (they read d_table)
  hipStream_t last_stream = nullptr;
  bool used = false;
  ~DevicePlan() {
    if (d_pieces) (void)hipFree(d_pieces);
    if (d_tasks) (void)hipFree(d_tasks);
    if (d_wide) (void)hipFree(d_wide);
    if (d_table) (void)hipFree(d_table);
    if (h_staging) (void)hipHostFree(h_staging);
    if (table_event) (void)hipEventDestroy(table_event);
    if (last_use) (void)hipEventDestroy(last_use);
  }
};

struct Workspace {
  void* ptr = nullptr;
  size_t bytes = 0;
  hipEvent_t last_use = nullptr;
  hipStream_t last_stream = nullptr;
  bool used = false;
};

struct TimingRec {
  costa_kernel_kind kind;
  hipEvent_t start, stop;
  int64_t bytes;
  int device;  // the device the events belong to
};

struct State {
  std::mutex mu;
  size_t workspace_limit = 0;
  std::map<std::string, std::unique_ptr<DevicePlan>> plans;
  std::map<std::string, std::unique_ptr<HostPlan>> host_plans;  // plan statistics without a device
  std::map<int, Workspace> ws;
  bool timing = false;
  std::vector<TimingRec> pending;
  std::map<int, std::vector<hipEvent_t>> event_pool;  // per device: events are recorded on that device's streams
  costa_timing totals{};
};

State& state() {
  static State* s = new State();
  return *s;
}

std::string plan_key(int device, int es, const std::vector<ItemDesc>& items, const std::vector<int32_t>& sigma,
                     size_t cap) {
  std::string k;
  auto put = [&](const void* p, size_t n) { k.append(reinterpret_cast<const char*>(p), n); };
  put(&device, sizeof device);
  put(&es, sizeof es);
  put(&cap, sizeof cap);
  size_t n = items.size();
  put(&n, sizeof n);
  for (const ItemDesc& d : items) {
    put(&d.A->id, sizeof d.A->id);
    put(&d.B->id, sizeof d.B->id);
    int32_t t = d.op == COSTA_OP_N ? 0 : 1;  // T and C move the same data
    put(&t, sizeof t);
    const char r = d.reads_a ? 1 : 0;  // stacks on A's side form only for pairs that do not read A
    put(&r, sizeof r);
  }
  size_t ns = sigma.size();
  put(&ns, sizeof ns);
  if (ns) put(sigma.data(), ns * sizeof(int32_t));
  return k;
}

PlanConfig make_config(int es) {
  PlanConfig c;
  c.elem_size = es;
  c.workspace_cap = INT64_MAX;
  c.max_piece_elems = kMaxPieceElems;
  return c;
}

// Validates a batch; fills `items` and `sig`.  No device calls.
bool is_zero(costa_dtype dt, const void* p);

costa_status validate(costa_dtype dtype, int32_t n, const costa_transform_desc* desc, const int32_t* sigma,
                      bool need_buffers, std::vector<ItemDesc>& items, std::vector<int32_t>& sig) {
  if (elem_size(dtype) == 0) return fail(COSTA_ERROR_INVALID_VALUE, "unknown dtype");
  if (n < 0) return fail(COSTA_ERROR_INVALID_VALUE, "negative batch size");
  if (n > 0 && !desc) return fail(COSTA_ERROR_INVALID_VALUE, "null descriptor array");
  if (n > 0xFFFF) return fail(COSTA_ERROR_NOT_SUPPORTED, "batch larger than 65535 pairs");
  items.clear();
  int32_t P = -1;
  for (int32_t k = 0; k < n; ++k) {
    const costa_transform_desc& d = desc[k];
    const Layout* A = layout_of(d.A);
    const Layout* B = layout_of(d.B);
    if (!A || !B) return fail(COSTA_ERROR_INVALID_VALUE, "null layout");
    if (d.op != COSTA_OP_N && d.op != COSTA_OP_T && d.op != COSTA_OP_C)
      return fail(COSTA_ERROR_INVALID_VALUE, "unknown op");
    const bool tr = d.op != COSTA_OP_N;
    if (A->nrows != (tr ? B->ncols : B->nrows) || A->ncols != (tr ? B->nrows : B->ncols))
      return fail(COSTA_ERROR_SHAPE_MISMATCH, "A is not the shape of op(B)");
    if (A->nranks != B->nranks) return fail(COSTA_ERROR_SHAPE_MISMATCH, "layouts of A and B have different P");
    if (P >= 0 && A->nranks != P) return fail(COSTA_ERROR_SHAPE_MISMATCH, "pairs of a batch have different P");
    P = A->nranks;
    if (A->nrows > INT32_MAX || A->ncols > INT32_MAX)
      return fail(COSTA_ERROR_NOT_SUPPORTED, "matrix dimension above 2^31-1");
    if (need_buffers) {
      if (!d.alpha || !d.beta) return fail(COSTA_ERROR_INVALID_VALUE, "null alpha or beta");
      if (!d.A_local || !d.B_local) return fail(COSTA_ERROR_INVALID_VALUE, "null buffer array");
    }
    // a missing beta (plan queries) counts as one that reads A
    items.push_back(ItemDesc{A, B, d.op, !(d.beta && is_zero(dtype, d.beta))});
  }
  sig.clear();
  if (sigma && P > 0) {
    std::vector<char> seen(P, 0);
    for (int32_t t = 0; t < P; ++t) {
      if (sigma[t] < 0 || sigma[t] >= P || seen[sigma[t]])
        return fail(COSTA_ERROR_INVALID_VALUE, "sigma is not a permutation of 0..P-1");
      seen[sigma[t]] = 1;
    }
    bool ident = true;
    for (int32_t t = 0; t < P; ++t) ident = ident && sigma[t] == t;
    if (!ident) sig.assign(sigma, sigma + P);
  }
  if (need_buffers) {
    for (int32_t k = 0; k < n; ++k) {
      const Layout* A = items[k].A;
      const Layout* B = items[k].B;
      for (int32_t t = 0; t < P; ++t) {
        int32_t r = sig.empty() ? t : sig[t];
        if (A->local_elems[t] > 0 && !desc[k].A_local[r])
          return fail(COSTA_ERROR_INVALID_VALUE, "null A buffer for a rank that holds data");
        if (B->local_elems[t] > 0 && !desc[k].B_local[t])
          return fail(COSTA_ERROR_INVALID_VALUE, "null B buffer for a rank that holds data");
      }
    }
  }
  return COSTA_SUCCESS;
}

bool is_zero(costa_dtype dt, const void* p) {
  if (dt == COSTA_R64) return *(const double*)p == 0.0;
  if (dt == COSTA_C128) return ((const double*)p)[0] == 0.0 && ((const double*)p)[1] == 0.0;
  if (dt == COSTA_R32) return *(const float*)p == 0.0f;
  return ((const float*)p)[0] == 0.0f && ((const float*)p)[1] == 0.0f;
}
bool is_one(costa_dtype dt, const void* p) {
  if (dt == COSTA_R64) return *(const double*)p == 1.0;
  if (dt == COSTA_C128) return ((const double*)p)[0] == 1.0 && ((const double*)p)[1] == 0.0;
  if (dt == COSTA_R32) return *(const float*)p == 1.0f;
  return ((const float*)p)[0] == 1.0f && ((const float*)p)[1] == 0.0f;
}
void to_pair(costa_dtype dt, const void* p, double out[2]) {
  out[0] = out[1] = 0.0;
  if (dt == COSTA_R64) out[0] = *(const double*)p;
  else if (dt == COSTA_C128) { out[0] = ((const double*)p)[0]; out[1] = ((const double*)p)[1]; }
  else if (dt == COSTA_R32) out[0] = *(const float*)p;
  else { out[0] = ((const float*)p)[0]; out[1] = ((const float*)p)[1]; }
}

// Timing events only measure: they skip the system-scope release (an L2
// write-back between the kernels they bracket), which the call's own ordering
// does not need.
#ifndef COSTA_TIMING_EVENT_FLAGS
#define COSTA_TIMING_EVENT_FLAGS hipEventDisableSystemFence
#endif

constexpr size_t kTimingEventsUpFront = 2048;

// A timing event of the current device (from its pool, else a new one).
hipEvent_t get_event(State& S, int device) {
  std::vector<hipEvent_t>& pool = S.event_pool[device];
  if (!pool.empty()) {
    hipEvent_t e = pool.back();
    pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, COSTA_TIMING_EVENT_FLAGS) != hipSuccess) return nullptr;
  return e;
}

void put_event(State& S, int device, hipEvent_t e) {
  if (e) S.event_pool[device].push_back(e);
}

costa_status collect_timing(State& S) {
  for (TimingRec& r : S.pending) {
    HIP_OR_FAIL(hipEventSynchronize(r.stop));
    float ms = 0.f;
    HIP_OR_FAIL(hipEventElapsedTime(&ms, r.start, r.stop));
    S.totals.ms[r.kind] += ms;
    S.totals.launches[r.kind] += 1;
    S.totals.bytes[r.kind] += r.bytes;
    put_event(S, r.device, r.start);
    put_event(S, r.device, r.stop);
  }
  S.pending.clear();
  return COSTA_SUCCESS;
}

// Device copies of a plan's tables (rectangles, task tables, wide task tables).
struct DeviceTables {
  const Piece* pieces;
  const int32_t* tasks;
  const int32_t* wide;
};

// Launches one mover range, bracketed by timing events when enabled (and
// `timed`).
costa_status run_range(State& S, MoverKind kind, costa_dtype dt, const DeviceTables& dt_, const LaunchRange& lr,
                       int32_t mode, int32_t conj, void* const* d_bufs, const ItemParam* d_items, int32_t allow_wide,
                       int64_t bytes, hipStream_t stream, bool timed = true) {
  if (lr.ntasks == 0) return COSTA_SUCCESS;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int device = 0;
  if (S.timing && timed) {
    if (S.pending.size() > 4096) {
      costa_status st = collect_timing(S);
      if (st != COSTA_SUCCESS) return st;
    }
    HIP_OR_FAIL(hipGetDevice(&device));
    e0 = get_event(S, device);
    e1 = get_event(S, device);
    if (!e0 || !e1) {
      put_event(S, device, e0);
      put_event(S, device, e1);
      return fail(COSTA_ERROR_DEVICE, "hipEventCreate failed");
    }
    HIP_OR_FAIL(hipEventRecord(e0, stream));
  }
  LaunchSpec spec{mode, conj, lr.has_transpose};
  HIP_OR_FAIL(launch_mover(kind, dt, spec, dt_.pieces, dt_.tasks + lr.task_begin, lr.ntasks,
                           lr.nwide ? dt_.wide + lr.wide_begin : nullptr, lr.nwide, d_bufs, d_items, allow_wide,
                           lr.xcd_ranges, stream));
  if (e1) {
    HIP_OR_FAIL(hipEventRecord(e1, stream));
    costa_kernel_kind kk = kind == KIND_PACK ? COSTA_KERNEL_PACK
                           : kind == KIND_UNPACK ? COSTA_KERNEL_UNPACK
                                                 : COSTA_KERNEL_DIRECT;
    S.pending.push_back(TimingRec{kk, e0, e1, bytes, device});
  }
  return COSTA_SUCCESS;
}

int64_t range_bytes(const LaunchRange& lr, int es, const std::vector<char>& reads_a) {
  int64_t b = 0;
  for (size_t k = 0; k < lr.item_elems.size(); ++k) b += lr.item_elems[k] * es * (2 + (reads_a[k] ? 1 : 0));
  return b;
}

// Message workspace of the current device, at least `bytes` large.
costa_status ensure_workspace(State& S, int device, size_t bytes, Workspace*& out) {
  Workspace& w = S.ws[device];
  out = &w;
  if (w.bytes >= bytes) return COSTA_SUCCESS;
  if (w.ptr) {
    HIP_OR_FAIL(hipDeviceSynchronize());
    HIP_OR_FAIL(hipFree(w.ptr));
    w.ptr = nullptr;
    w.bytes = 0;
  }
  if (bytes == 0) return COSTA_SUCCESS;
  hipError_t e = hipMalloc(&w.ptr, bytes);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    w.ptr = nullptr;
    return fail(COSTA_ERROR_OUT_OF_MEMORY, "cannot allocate " + std::to_string(bytes) + " bytes of message workspace");
  }
  w.bytes = bytes;
  if (!w.last_use) HIP_OR_FAIL(hipEventCreateWithFlags(&w.last_use, hipEventDisableTiming));
  return COSTA_SUCCESS;
}

int64_t auto_cap(State& S, int device, int64_t needed) {
  if (S.workspace_limit) return std::min<int64_t>(needed, (int64_t)S.workspace_limit);
  size_t free_b = 0, total_b = 0;
  if (hipMemGetInfo(&free_b, &total_b) != hipSuccess) {
    (void)hipGetLastError();
    return needed;
  }
  int64_t have = (int64_t)S.ws[device].bytes + (int64_t)free_b;  // the current workspace can be reused
  int64_t cap = (int64_t)(0.6 * (double)have);
  cap = std::max<int64_t>(cap, 64ll << 20);
  return std::min(needed, cap);
}

costa_status get_plan(State& S, costa_dtype dt, const std::vector<ItemDesc>& items, const std::vector<int32_t>& sig,
                      DevicePlan*& out) {
  int device = 0;
  HIP_OR_FAIL(hipGetDevice(&device));
  const int es = elem_size(dt);
  std::string key = plan_key(device, es, items, sig, S.workspace_limit);
  auto it = S.plans.find(key);
  if (it != S.plans.end()) {
    out = it->second.get();
    return COSTA_SUCCESS;
  }
  if (S.plans.size() >= 32) {  // bounded cache: drop everything (plans are cheap to rebuild)
    HIP_OR_FAIL(hipDeviceSynchronize());
    S.plans.clear();
  }
  std::unique_ptr<DevicePlan> dp(new (std::nothrow) DevicePlan());
  if (!dp) return fail(COSTA_ERROR_OUT_OF_MEMORY, "host allocation failed");
  dp->device = device;
  PlanConfig cfg = make_config(es);
  try {
    build_plan(items, sig, cfg, [&](int64_t need) { return auto_cap(S, device, need); }, dp->host);
  } catch (const std::bad_alloc&) {
    return fail(COSTA_ERROR_OUT_OF_MEMORY, "host allocation failed while planning");
  }
  const HostPlan& hp = dp->host;
  if (!hp.pieces.empty()) {
    HIP_OR_FAIL(hipMalloc(&dp->d_pieces, hp.pieces.size() * sizeof(Piece)));
    HIP_OR_FAIL(hipMemcpy(dp->d_pieces, hp.pieces.data(), hp.pieces.size() * sizeof(Piece), hipMemcpyHostToDevice));
    HIP_OR_FAIL(hipMalloc(&dp->d_tasks, hp.tasks.size() * sizeof(int32_t)));
    HIP_OR_FAIL(hipMemcpy(dp->d_tasks, hp.tasks.data(), hp.tasks.size() * sizeof(int32_t), hipMemcpyHostToDevice));
    if (!hp.wide_tasks.empty()) {
      HIP_OR_FAIL(hipMalloc(&dp->d_wide, hp.wide_tasks.size() * sizeof(int32_t)));
      HIP_OR_FAIL(hipMemcpy(dp->d_wide, hp.wide_tasks.data(), hp.wide_tasks.size() * sizeof(int32_t),
                            hipMemcpyHostToDevice));
    }
  }
  const int32_t P = items.empty() ? 0 : items[0].A->nranks;
  dp->nbufs = (size_t)2 * items.size() * P + 1;
  size_t ptr_bytes = (dp->nbufs * sizeof(void*) + 63) / 64 * 64;
  dp->table_bytes = ptr_bytes + items.size() * sizeof(ItemParam);
  HIP_OR_FAIL(hipMalloc(&dp->d_table, dp->table_bytes));
  HIP_OR_FAIL(hipHostMalloc(&dp->h_staging, dp->table_bytes, hipHostMallocDefault));
  HIP_OR_FAIL(hipEventCreateWithFlags(&dp->table_event, hipEventDisableTiming));
  HIP_OR_FAIL(hipEventCreateWithFlags(&dp->last_use, hipEventDisableTiming));
  out = dp.get();
  S.plans.emplace(key, std::move(dp));
  return COSTA_SUCCESS;
}

// The table a call's kernels read: the buffer pointers (A of pair k, rank r
// at k*P + r; B at n*P + k*P + s; the message workspace at 2*n*P), padded to
// 64 bytes, then one ItemParam per pair.  Returns the pointers' byte size;
// reads_a[k]: pair k reads A (beta != 0); aligned: every buffer 16-byte
// aligned.
size_t call_table(costa_dtype dt, int32_t n, const costa_transform_desc* desc, int32_t P, void* messages,
                  std::vector<unsigned char>& table, std::vector<char>& reads_a, bool& aligned) {
  const size_t nbufs = (size_t)2 * n * P + 1;
  const size_t ptr_bytes = (nbufs * sizeof(void*) + 63) / 64 * 64;
  table.assign(ptr_bytes + (size_t)n * sizeof(ItemParam), 0);
  void** bp = reinterpret_cast<void**>(table.data());
  aligned = true;
  auto note = [&](const void* p) { aligned = aligned && ((uintptr_t)p % 16 == 0); };
  for (int32_t k = 0; k < n; ++k)
    for (int32_t r = 0; r < P; ++r) {
      bp[(size_t)k * P + r] = desc[k].A_local[r];
      bp[(size_t)n * P + (size_t)k * P + r] = const_cast<void*>(desc[k].B_local[r]);
      note(desc[k].A_local[r]);
      note(desc[k].B_local[r]);
    }
  bp[(size_t)2 * n * P] = messages;
  ItemParam* ipar = reinterpret_cast<ItemParam*>(table.data() + ptr_bytes);
  reads_a.assign(n, 0);
  for (int32_t k = 0; k < n; ++k) {
    ItemParam& q = ipar[k];
    to_pair(dt, desc[k].alpha, q.alpha);
    to_pair(dt, desc[k].beta, q.beta);
    const bool bz = is_zero(dt, desc[k].beta);
    q.mode = bz ? (is_one(dt, desc[k].alpha) ? MODE_COPY : MODE_SCALE) : MODE_AXPBY;
    q.conj = (desc[k].op == COSTA_OP_C && is_complex(dt)) ? 1 : 0;
    reads_a[k] = !bz;
  }
  return ptr_bytes;
}

// Enqueues every launch of a plan: the direct path (when not merged), then
// pack and unpack-transform of each wave.
costa_status launch_plan(State& S, costa_dtype dt, const HostPlan& hp, const DeviceTables& tabs,
                         const ItemParam* ipar, int32_t n, const std::vector<char>& reads_a, bool aligned,
                         void* const* d_bufs, const ItemParam* d_items, hipStream_t stream, bool timed) {
  const int es = elem_size(dt);
  const int32_t wide = aligned ? 1 : 0;
  // one arithmetic mode for the whole call when every pair agrees
  int32_t mode = ipar[0].mode, conj = ipar[0].conj;
  for (int32_t k = 1; k < n; ++k)
    if (ipar[k].mode != mode || ipar[k].conj != conj) mode = -1;
  costa_status st;
  for (const LaunchRange& lr : hp.direct) {
    st = run_range(S, KIND_DIRECT, dt, tabs, lr, mode, conj, d_bufs, d_items, wide, range_bytes(lr, es, reads_a),
                   stream, timed);
    if (st != COSTA_SUCCESS) return st;
  }
  std::vector<char> no_read(n, 0);
  for (const Wave& w : hp.waves) {
    st = run_range(S, KIND_PACK, dt, tabs, w.pack, MODE_COPY, 0, d_bufs, d_items, wide,
                   range_bytes(w.pack, es, no_read), stream, timed);
    if (st != COSTA_SUCCESS) return st;
    for (const LaunchRange& lr : w.unpack) {
      st = run_range(S, KIND_UNPACK, dt, tabs, lr, mode, conj, d_bufs, d_items, wide, range_bytes(lr, es, reads_a),
                     stream, timed);
      if (st != COSTA_SUCCESS) return st;
    }
  }
  return COSTA_SUCCESS;
}

costa_status transform_impl(costa_dtype dt, int32_t n, const costa_transform_desc* desc, const int32_t* sigma,
                            hipStream_t stream) {
  State& S = state();
  std::vector<ItemDesc> items;
  std::vector<int32_t> sig;
  costa_status st = validate(dt, n, desc, sigma, true, items, sig);
  if (st != COSTA_SUCCESS) return st;
  std::lock_guard<std::mutex> lock(S.mu);
  int64_t total = 0;
  for (const ItemDesc& d : items) total += d.A->nrows * d.A->ncols;
  if (total == 0) return COSTA_SUCCESS;
  DevicePlan* dp = nullptr;
  st = get_plan(S, dt, items, sig, dp);
  if (st != COSTA_SUCCESS) return st;
  const HostPlan& hp = dp->host;
  const int32_t P = items[0].A->nranks;

  Workspace* ws = nullptr;
  st = ensure_workspace(S, dp->device, (size_t)hp.workspace_bytes, ws);
  if (st != COSTA_SUCCESS) return st;

  std::vector<unsigned char> table;
  std::vector<char> reads_a;
  bool aligned = true;
  const size_t ptr_bytes = call_table(dt, n, desc, P, ws->ptr, table, reads_a, aligned);
  if (table != dp->last_table) {
    // the kernels of the plan's last call read the table until they end: on
    // another stream, the new table is written only after them
    if (dp->used && dp->last_stream != stream) HIP_OR_FAIL(hipStreamWaitEvent(stream, dp->last_use, 0));
    if (dp->table_pending) HIP_OR_FAIL(hipEventSynchronize(dp->table_event));
    std::memcpy(dp->h_staging, table.data(), table.size());
    HIP_OR_FAIL(hipMemcpyAsync(dp->d_table, dp->h_staging, table.size(), hipMemcpyHostToDevice, stream));
    HIP_OR_FAIL(hipEventRecord(dp->table_event, stream));
    dp->table_pending = true;
    dp->last_table.swap(table);
  }
  // message buffers are shared by every call on this device: order after the last user
  if (ws->used && ws->last_stream != stream) HIP_OR_FAIL(hipStreamWaitEvent(stream, ws->last_use, 0));

  void* const* d_bufs = reinterpret_cast<void* const*>(dp->d_table);
  const ItemParam* d_items = reinterpret_cast<const ItemParam*>((unsigned char*)dp->d_table + ptr_bytes);
  const ItemParam* ipar = reinterpret_cast<const ItemParam*>(dp->last_table.data() + ptr_bytes);
  st = launch_plan(S, dt, hp, DeviceTables{dp->d_pieces, dp->d_tasks, dp->d_wide}, ipar, n, reads_a, aligned,
                   d_bufs, d_items, stream, true);
  if (st != COSTA_SUCCESS) return st;
  if (ws->last_use) {
    HIP_OR_FAIL(hipEventRecord(ws->last_use, stream));
    ws->last_stream = stream;
    ws->used = true;
  }
  HIP_OR_FAIL(hipEventRecord(dp->last_use, stream));
  dp->last_stream = stream;
  dp->used = true;
  return COSTA_SUCCESS;
}

}  // namespace
}  // namespace costa

using namespace costa;

extern "C" costa_status costa_transform(costa_dtype dtype, costa_op op, const void* alpha, const void* beta,
                                        costa_layout A, void* const* A_local, costa_layout B,
                                        const void* const* B_local, const int32_t* sigma, hipStream_t stream) {
  return guarded([&]() -> costa_status {
    costa_transform_desc d{op, alpha, beta, A, A_local, B, B_local};
    return transform_impl(dtype, 1, &d, sigma, stream);
  });
}

extern "C" costa_status costa_transform_batched(costa_dtype dtype, int32_t n, const costa_transform_desc* desc,
                                                const int32_t* sigma, hipStream_t stream) {
  return guarded([&]() -> costa_status {
    return transform_impl(dtype, n, desc, sigma, stream);
  });
}

extern "C" costa_status costa_set_workspace_limit(size_t bytes) {
  return guarded([&]() -> costa_status {
    State& S = state();
    std::lock_guard<std::mutex> lock(S.mu);
    S.workspace_limit = bytes;
    return COSTA_SUCCESS;
  });
}

// Host-only plan (no device): the workspace cap is the user limit, else unlimited.
costa_status host_plan(costa_dtype dtype, int32_t n, const costa_transform_desc* desc, const int32_t* sigma,
                       const HostPlan*& out) {
  std::vector<ItemDesc> items;
  std::vector<int32_t> sig;
  costa_status st = validate(dtype, n, desc, sigma, false, items, sig);
  if (st != COSTA_SUCCESS) return st;
  State& S = state();
  const int es = elem_size(dtype);
  std::string key = plan_key(-1, es, items, sig, S.workspace_limit);
  auto it = S.host_plans.find(key);
  if (it == S.host_plans.end()) {
    if (S.host_plans.size() >= 32) S.host_plans.clear();
    std::unique_ptr<HostPlan> hp(new (std::nothrow) HostPlan());
    if (!hp) return fail(COSTA_ERROR_OUT_OF_MEMORY, "host allocation failed");
    PlanConfig cfg = make_config(es);
    size_t lim = S.workspace_limit;
    try {
      build_plan(items, sig, cfg, [lim](int64_t need) { return lim ? std::min<int64_t>(need, (int64_t)lim) : need; },
                 *hp);
    } catch (const std::bad_alloc&) {
      return fail(COSTA_ERROR_OUT_OF_MEMORY, "host allocation failed while planning");
    }
    it = S.host_plans.emplace(key, std::move(hp)).first;
  }
  out = it->second.get();
  return COSTA_SUCCESS;
}

extern "C" costa_status costa_plan_export(costa_dtype dtype, int32_t n, const costa_transform_desc* desc,
                                          const int32_t* sigma, costa_piece_info* out, int64_t capacity,
                                          int64_t* count) {
  return guarded([&]() -> costa_status {
    if (!count || capacity < 0 || (capacity > 0 && !out)) return fail(COSTA_ERROR_INVALID_VALUE, "bad output array");
    State& S = state();
    std::lock_guard<std::mutex> lock(S.mu);
    const HostPlan* hp = nullptr;
    costa_status st = host_plan(dtype, n, desc, sigma, hp);
    if (st != COSTA_SUCCESS) return st;
    int64_t k = 0;
    int32_t launch = 0;
    auto emit = [&](const LaunchRange& lr, costa_kernel_kind kind, int32_t wave) {
      for (int64_t i = 0; i < lr.npieces; ++i, ++k) {
        if (k >= capacity) continue;
        const Piece& q = hp->pieces[lr.piece_begin + i];
        // workgroups that move it: from task0 up to the next rectangle's first
        // one (or the launch's end); 1 for a rectangle that shares a workgroup
        int64_t end = lr.ntasks;
        for (int64_t j = i + 1; j < lr.npieces; ++j)
          if (hp->pieces[lr.piece_begin + j].task0 != q.task0) {
            end = hp->pieces[lr.piece_begin + j].task0;
            break;
          }
        costa_piece_info& o = out[k];
        o.kind = kind;
        o.wave = wave;
        o.group = q.task0;
        o.src_off = q.src_off;
        o.dst_off = q.dst_off;
        o.src_ld = q.src_ld;
        o.dst_ld = q.dst_ld;
        o.src_buf = q.src_buf;
        o.dst_buf = q.dst_buf;
        o.nx = q.nx;
        o.ny = q.ny;
        o.item = q.item;
        o.flags = q.flags;
        o.ntasks = end - q.task0;
        const bool T = q.flags & PIECE_TRANSPOSE;
        o.tile_x = T ? tile_x_of(q.aux) : 0;
        o.tile_y = T ? tile_y_of(q.aux) : 0;
        // its first task and task count in the wide table (launches without tiles)
        o.wide_group = lr.nwide ? q.aux : -1;
        int64_t wend = lr.nwide;
        for (int64_t j = i + 1; lr.nwide && j < lr.npieces; ++j)
          if (hp->pieces[lr.piece_begin + j].aux != q.aux) {
            wend = hp->pieces[lr.piece_begin + j].aux;
            break;
          }
        o.wide_ntasks = lr.nwide ? wend - q.aux : 0;
        o.launch = launch;
        o.reserved = 0;

      }
      ++launch;
    };
    for (const LaunchRange& lr : hp->direct) emit(lr, COSTA_KERNEL_DIRECT, 0);
    for (size_t w = 0; w < hp->waves.size(); ++w) {
      emit(hp->waves[w].pack, COSTA_KERNEL_PACK, (int32_t)w);
      for (const LaunchRange& lr : hp->waves[w].unpack) emit(lr, COSTA_KERNEL_UNPACK, (int32_t)w);
    }
    *count = k;
    return COSTA_SUCCESS;
  });
}

extern "C" costa_status costa_plan_stats(costa_dtype dtype, int32_t n, const costa_transform_desc* desc,
                                         const int32_t* sigma, costa_stats* out) {
  return guarded([&]() -> costa_status {
    if (!out) return fail(COSTA_ERROR_INVALID_VALUE, "null output");
    State& S = state();
    std::lock_guard<std::mutex> lock(S.mu);
    const HostPlan* hpp = nullptr;
    costa_status st = host_plan(dtype, n, desc, sigma, hpp);
    if (st != COSTA_SUCCESS) return st;
    const HostPlan& hp = *hpp;
    const int es = elem_size(dtype);
    costa_stats s{};
    s.overlay_blocks = hp.overlay_blocks;
    for (int32_t k = 0; k < n; ++k) {
      bool reads_a = !(desc[k].beta && is_zero(dtype, desc[k].beta));
      s.total_elems += hp.item_total[k];
      s.local_elems += hp.item_local[k];
      s.remote_elems += hp.item_remote[k];
      s.model_bytes += (int64_t)es * (hp.item_total[k] * (2 + (reads_a ? 1 : 0)) + 2 * hp.item_remote[k]);
      s.pack_bytes += (int64_t)es * 2 * hp.item_remote[k];
      s.unpack_bytes += (int64_t)es * hp.item_remote[k] * (2 + (reads_a ? 1 : 0));
      s.direct_bytes += (int64_t)es * hp.item_local[k] * (2 + (reads_a ? 1 : 0));
    }
    s.message_bytes = (int64_t)es * s.remote_elems;
    s.workspace_bytes = hp.workspace_bytes;
    s.waves = (int32_t)hp.waves.size();
    s.pieces_pack = hp.pieces_pack;
    s.pieces_unpack = hp.pieces_unpack;
    s.pieces_direct = hp.pieces_direct;
    s.plan_ms = hp.plan_ms;
    *out = s;
    return COSTA_SUCCESS;
  });
}

namespace costa {
namespace {

// Device allocation released when it goes out of scope.
struct DevBuf {
  void* p = nullptr;
  DevBuf() = default;
  DevBuf(const DevBuf&) = delete;
  DevBuf& operator=(const DevBuf&) = delete;
  ~DevBuf() {
    if (p) (void)hipFree(p);
  }
  hipError_t alloc(size_t n) { return hipMalloc(&p, n ? n : 1); }
  template <typename T>
  T* as() const {
    return reinterpret_cast<T*>(p);
  }
};

// Uploads `n` items of `src` into a fresh device buffer on `stream`.
template <typename T>
hipError_t upload(DevBuf& d, const T* src, size_t n, hipStream_t stream) {
  hipError_t e = d.alloc(n * sizeof(T));
  if (e != hipSuccess || n == 0) return e;
  return hipMemcpyAsync(d.p, src, n * sizeof(T), hipMemcpyHostToDevice, stream);
}

}  // namespace
}  // namespace costa

extern "C" costa_status costa_volume_matrix(costa_layout A_h, costa_layout B_h, costa_op op, int64_t* V_host,
                                            hipStream_t stream) {
  return guarded([&]() -> costa_status {
    const Layout* A = layout_of(A_h);
    const Layout* B = layout_of(B_h);
    if (!A || !B || !V_host) return fail(COSTA_ERROR_INVALID_VALUE, "null argument");
    if (op != COSTA_OP_N && op != COSTA_OP_T && op != COSTA_OP_C) return fail(COSTA_ERROR_INVALID_VALUE, "unknown op");
    const bool tr = op != COSTA_OP_N;
    if (A->nrows != (tr ? B->ncols : B->nrows) || A->ncols != (tr ? B->nrows : B->ncols))
      return fail(COSTA_ERROR_SHAPE_MISMATCH, "A is not the shape of op(B)");
    if (A->nranks != B->nranks) return fail(COSTA_ERROR_SHAPE_MISMATCH, "layouts of A and B have different P");
    const int32_t P = A->nranks;
    const size_t PP = (size_t)P * P;
    std::memset(V_host, 0, sizeof(int64_t) * PP);
    std::vector<Interval> rows = overlay(A->rsplit, tr ? B->csplit : B->rsplit);
    std::vector<Interval> cols = overlay(A->csplit, tr ? B->rsplit : B->csplit);
    if (rows.empty() || cols.empty()) return COSTA_SUCCESS;
    if (rows.size() > INT32_MAX || cols.size() > INT32_MAX)
      return fail(COSTA_ERROR_NOT_SUPPORTED, "more than 2^31 overlay intervals in one dimension");
    State& S = state();
    std::lock_guard<std::mutex> lock(S.mu);
    // two block-cyclic layouts (with or without a rank map): the separable kernels
    const bool separable = A->block_cyclic && B->block_cyclic;
    DevBuf d_rows, d_cols, d_oa, d_ob, d_v, d_hr, d_hc, d_ca, d_cb;
    std::vector<unsigned long long> zeros;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    int ev_device = 0;
    if (S.timing && hipGetDevice(&ev_device) == hipSuccess) {
      e0 = get_event(S, ev_device);
      e1 = get_event(S, ev_device);
    }
    auto run = [&]() -> costa_status {
      HIP_OR_FAIL(d_v.alloc(sizeof(int64_t) * PP));
      if (separable) {
        // classes of the covering blocks: process row/column of A's block and
        // of op(B)'s block (B's process column for the rows of op(B) when
        // transposed, and its process row for the columns)
        const int32_t nrb = tr ? B->pcol : B->prow, ncb = tr ? B->prow : B->pcol;
        for (Interval& v : rows) {
          v.a = A->prow_of(v.a);
          v.b = tr ? B->pcol_of(v.b) : B->prow_of(v.b);
        }
        for (Interval& v : cols) {
          v.a = A->pcol_of(v.a);
          v.b = tr ? B->prow_of(v.b) : B->pcol_of(v.b);
        }
        const size_t nh_r = (size_t)nrb * A->prow, nh_c = (size_t)ncb * A->pcol;
        zeros.assign(std::max(nh_r, nh_c), 0ull);
        // each rank's row and column class in A's grid and in op(B)'s (-1
        // outside the grid: a rank map may leave ranks out)
        std::vector<int32_t> ca((size_t)2 * P, -1), cb((size_t)2 * P, -1);
        for (int32_t pr = 0; pr < A->prow; ++pr)
          for (int32_t pc = 0; pc < A->pcol; ++pc) {
            const int32_t r = A->rank_at(pr, pc);
            ca[(size_t)2 * r] = pr;
            ca[(size_t)2 * r + 1] = pc;
          }
        for (int32_t pr = 0; pr < B->prow; ++pr)
          for (int32_t pc = 0; pc < B->pcol; ++pc) {
            const int32_t r = B->rank_at(pr, pc);
            cb[(size_t)2 * r] = tr ? pc : pr;
            cb[(size_t)2 * r + 1] = tr ? pr : pc;
          }
        HIP_OR_FAIL(upload(d_rows, rows.data(), rows.size(), stream));
        HIP_OR_FAIL(upload(d_cols, cols.data(), cols.size(), stream));
        HIP_OR_FAIL(upload(d_hr, zeros.data(), nh_r, stream));
        HIP_OR_FAIL(upload(d_hc, zeros.data(), nh_c, stream));
        HIP_OR_FAIL(upload(d_ca, ca.data(), ca.size(), stream));
        HIP_OR_FAIL(upload(d_cb, cb.data(), cb.size(), stream));
        SeparableArgs a{d_rows.as<Interval>(), (int32_t)rows.size(), d_cols.as<Interval>(), (int32_t)cols.size(),
                        nrb, A->prow, ncb, A->pcol, d_hr.as<unsigned long long>(), d_hc.as<unsigned long long>(),
                        d_ca.as<int32_t>(), d_cb.as<int32_t>(), P, d_v.as<unsigned long long>()};
        if (e0) HIP_OR_FAIL(hipEventRecord(e0, stream));
        HIP_OR_FAIL(launch_volume_separable(a, stream));
      } else {
        // owner tables (block-cyclic layouts keep none: write them out here)
        std::vector<int32_t> oa_tmp, ob_tmp;
        auto owners = [](const Layout* L, std::vector<int32_t>& tmp) -> const std::vector<int32_t>& {
          if (!L->block_cyclic) return L->owner;
          tmp.resize((size_t)L->nbr * L->nbc);
          for (int32_t bi = 0; bi < L->nbr; ++bi)
            for (int32_t bj = 0; bj < L->nbc; ++bj) tmp[L->block(bi, bj)] = L->owner_of(bi, bj);
          return tmp;
        };
        const std::vector<int32_t>& oa = owners(A, oa_tmp);
        const std::vector<int32_t>& ob = owners(B, ob_tmp);
        zeros.assign(PP, 0ull);
        HIP_OR_FAIL(upload(d_rows, rows.data(), rows.size(), stream));
        HIP_OR_FAIL(upload(d_cols, cols.data(), cols.size(), stream));
        HIP_OR_FAIL(upload(d_oa, oa.data(), oa.size(), stream));
        HIP_OR_FAIL(upload(d_ob, ob.data(), ob.size(), stream));
        HIP_OR_FAIL(hipMemcpyAsync(d_v.p, zeros.data(), sizeof(int64_t) * PP, hipMemcpyHostToDevice, stream));
        VolumeArgs a{d_rows.as<Interval>(), (int32_t)rows.size(), d_cols.as<Interval>(), (int32_t)cols.size(),
                     d_oa.as<int32_t>(), A->nbc, d_ob.as<int32_t>(), B->nbc, tr ? 1 : 0, P,
                     d_v.as<unsigned long long>()};
        if (e0) HIP_OR_FAIL(hipEventRecord(e0, stream));
        HIP_OR_FAIL(launch_volume(a, stream));
      }
      if (e1) {
        HIP_OR_FAIL(hipEventRecord(e1, stream));
        S.pending.push_back(
            TimingRec{COSTA_KERNEL_VOLUME, e0, e1, (int64_t)(rows.size() + cols.size()) * 24, ev_device});
        e0 = e1 = nullptr;
      }
      HIP_OR_FAIL(hipMemcpyAsync(V_host, d_v.p, sizeof(int64_t) * PP, hipMemcpyDeviceToHost, stream));
      HIP_OR_FAIL(hipStreamSynchronize(stream));
      return COSTA_SUCCESS;
    };
    costa_status st = run();
    (void)hipStreamSynchronize(stream);  // device buffers are freed below
    put_event(S, ev_device, e0);
    put_event(S, ev_device, e1);
    return st;
  });
}

// ---------------------------------------------------------------------------
// The transform that allocates nothing
// ---------------------------------------------------------------------------
namespace costa {
namespace {

constexpr size_t kNoallocBytes = COSTA_NOALLOC_SCRATCH_BYTES;
constexpr size_t kNoallocTableBytes = COSTA_NOALLOC_TABLE_BYTES;
constexpr size_t kNoallocMessageBytes = kNoallocBytes - kNoallocTableBytes;
static_assert(kNoallocTableBytes % 256 == 0 && kNoallocTableBytes < kNoallocBytes, "scratch partition");

// The device memory of costa_transform_batched_noalloc: the plan's tables and
// the call's pointer table in the first kNoallocTableBytes, the message
// buffers of one wave in the rest.  Each device holds its own copy until the
// process ends.  In host code this name is only a stand-in: host code uses
// the address hipGetSymbolAddress returns on each device.
static __device__ __align__(256) unsigned char scratch[kNoallocBytes];

// A plan of the no-allocation path: planned for messages of at most
// kNoallocMessageBytes per wave, with the offsets of its tables in the
// scratch array.
struct NoallocPlan {
  HostPlan host;
  uint64_t serial = 0;  // tells plans apart when one is rebuilt at a freed address
  size_t off_tasks = 0, off_wide = 0, off_table = 0, end = 0;
};

// What one device's scratch array holds.
struct NoallocDevice {
  unsigned char* base = nullptr;     // address of `scratch` on the device
  uint64_t resident = 0;             // serial of the plan whose tables it holds (0: none)
  std::vector<unsigned char> table;  // the call table it holds
};

struct NoallocState {
  std::map<std::string, std::unique_ptr<NoallocPlan>> plans;
  std::map<int, NoallocDevice> devices;
  uint64_t next_serial = 1;
};

NoallocState& noalloc_state() {
  static NoallocState* s = new NoallocState();
  return *s;
}

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

// Host plan of a no-allocation call (host memory only; no device call).
costa_status noalloc_plan(costa_dtype dt, const std::vector<ItemDesc>& items, const std::vector<int32_t>& sig,
                          NoallocPlan*& out) {
  NoallocState& N = noalloc_state();
  const int es = elem_size(dt);
  std::string key = plan_key(-1, es, items, sig, kNoallocMessageBytes);
  auto it = N.plans.find(key);
  if (it == N.plans.end()) {
    if (N.plans.size() >= 32) N.plans.clear();
    std::unique_ptr<NoallocPlan> np(new NoallocPlan());
    build_plan(items, sig, make_config(es),
               [](int64_t need) { return std::min<int64_t>(need, (int64_t)kNoallocMessageBytes); }, np->host);
    const HostPlan& hp = np->host;
    const int32_t P = items.empty() ? 0 : items[0].A->nranks;
    const size_t nbufs = (size_t)2 * items.size() * P + 1;
    np->off_tasks = align256(hp.pieces.size() * sizeof(Piece));
    np->off_wide = np->off_tasks + align256(hp.tasks.size() * sizeof(int32_t));
    np->off_table = np->off_wide + align256(hp.wide_tasks.size() * sizeof(int32_t));
    np->end = np->off_table + (nbufs * sizeof(void*) + 63) / 64 * 64 + items.size() * sizeof(ItemParam);
    np->serial = N.next_serial++;
    it = N.plans.emplace(key, std::move(np)).first;
  }
  NoallocPlan& np = *it->second;
  if (np.end > kNoallocTableBytes)
    return fail(COSTA_ERROR_NOT_SUPPORTED, "the plan's tables need " + std::to_string(np.end) +
                                               " bytes; the no-allocation scratch holds " +
                                               std::to_string(kNoallocTableBytes) +
                                               " bytes of tables (costa_transform_batched has no such limit)");
  if ((size_t)np.host.workspace_bytes > kNoallocMessageBytes)
    return fail(COSTA_ERROR_NOT_SUPPORTED, "a wave's messages exceed the no-allocation scratch");
  out = &np;
  return COSTA_SUCCESS;
}

// The scratch array of the current device: its address, looked up once per
// device with that device current.
costa_status noalloc_device(NoallocDevice*& out) {
  int device = 0;
  HIP_OR_FAIL(hipGetDevice(&device));
  NoallocDevice& d = noalloc_state().devices[device];
  if (!d.base) {
    void* ptr = nullptr;
    HIP_OR_FAIL(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
    if (!ptr || (uintptr_t)ptr % 256 != 0) return fail(COSTA_ERROR_DEVICE, "scratch array address is not usable");
    d.base = static_cast<unsigned char*>(ptr);
  }
  out = &d;
  return COSTA_SUCCESS;
}

}  // namespace
}  // namespace costa

extern "C" costa_status costa_transform_batched_noalloc(costa_dtype dtype, int32_t n, const costa_transform_desc* desc,
                                                        const int32_t* sigma, hipStream_t stream) {
  return guarded([&]() -> costa_status {
    std::vector<ItemDesc> items;
    std::vector<int32_t> sig;
    costa_status st = validate(dtype, n, desc, sigma, true, items, sig);
    if (st != COSTA_SUCCESS) return st;
    State& S = state();
    std::lock_guard<std::mutex> lock(S.mu);
    int64_t total = 0;
    for (const ItemDesc& d : items) total += d.A->nrows * d.A->ncols;
    if (total == 0) return COSTA_SUCCESS;
    // planning and the size checks come first: a request that does not fit
    // is refused before any device call
    NoallocPlan* np = nullptr;
    st = noalloc_plan(dtype, items, sig, np);
    if (st != COSTA_SUCCESS) return st;
    NoallocDevice* dev = nullptr;
    st = noalloc_device(dev);
    if (st != COSTA_SUCCESS) return st;
    const HostPlan& hp = np->host;
    unsigned char* base = dev->base;
    // the plan's tables, unless the scratch holds them already (copies from
    // pageable host memory: the host data has been taken when the call returns)
    if (dev->resident != np->serial) {
      dev->resident = 0;
      dev->table.clear();
      if (!hp.pieces.empty())
        HIP_OR_FAIL(hipMemcpyAsync(base, hp.pieces.data(), hp.pieces.size() * sizeof(Piece), hipMemcpyHostToDevice,
                                   stream));
      if (!hp.tasks.empty())
        HIP_OR_FAIL(hipMemcpyAsync(base + np->off_tasks, hp.tasks.data(), hp.tasks.size() * sizeof(int32_t),
                                   hipMemcpyHostToDevice, stream));
      if (!hp.wide_tasks.empty())
        HIP_OR_FAIL(hipMemcpyAsync(base + np->off_wide, hp.wide_tasks.data(), hp.wide_tasks.size() * sizeof(int32_t),
                                   hipMemcpyHostToDevice, stream));
      dev->resident = np->serial;
    }
    const int32_t P = items[0].A->nranks;
    std::vector<unsigned char> table;
    std::vector<char> reads_a;
    bool aligned = true;
    const size_t ptr_bytes = call_table(dtype, n, desc, P, base + kNoallocTableBytes, table, reads_a, aligned);
    if (table != dev->table) {
      HIP_OR_FAIL(hipMemcpyAsync(base + np->off_table, table.data(), table.size(), hipMemcpyHostToDevice, stream));
      dev->table.swap(table);
    }
    const ItemParam* ipar = reinterpret_cast<const ItemParam*>(dev->table.data() + ptr_bytes);
    void* const* d_bufs = reinterpret_cast<void* const*>(base + np->off_table);
    const ItemParam* d_items = reinterpret_cast<const ItemParam*>(base + np->off_table + ptr_bytes);
    const DeviceTables tabs{reinterpret_cast<const Piece*>(base),
                            reinterpret_cast<const int32_t*>(base + np->off_tasks),
                            reinterpret_cast<const int32_t*>(base + np->off_wide)};
    // no timing events on this path (creating one may allocate)
    return launch_plan(S, dtype, hp, tabs, ipar, n, reads_a, aligned, d_bufs, d_items, stream, false);
  });
}

extern "C" costa_status costa_timing_enable(int on) {
  return guarded([&]() -> costa_status {
    State& S = state();
    std::lock_guard<std::mutex> lock(S.mu);
    costa_status st = collect_timing(S);
    S.timing = on != 0;
    S.totals = costa_timing{};
    // create the events up front (hipEventCreate can take tens of
    // microseconds; created lazily, they would land in the timed calls)
    int dev = 0;
    if (st == COSTA_SUCCESS && S.timing && hipGetDevice(&dev) == hipSuccess) {
      std::vector<hipEvent_t>& pool = S.event_pool[dev];
      while (pool.size() < kTimingEventsUpFront) {
        hipEvent_t e = nullptr;
        if (hipEventCreateWithFlags(&e, COSTA_TIMING_EVENT_FLAGS) != hipSuccess) break;
        pool.push_back(e);
      }
    }
    return st;
  });
}

extern "C" costa_status costa_timing_read(costa_timing* out) {
  return guarded([&]() -> costa_status {
    if (!out) return fail(COSTA_ERROR_INVALID_VALUE, "null output");
    State& S = state();
    std::lock_guard<std::mutex> lock(S.mu);
    costa_status st = collect_timing(S);
    *out = S.totals;
    return st;
  });
}

extern "C" costa_status costa_finalize(void) {
  return guarded([&]() -> costa_status {
    State& S = state();
    {
      std::lock_guard<std::mutex> lock(S.mu);
      NoallocState& N = noalloc_state();
      if (!S.plans.empty() || !S.ws.empty() || !S.pending.empty() || !N.devices.empty())
        HIP_OR_FAIL(hipDeviceSynchronize());
      for (const TimingRec& r : S.pending) {  // recorded but never read: their events go too
        (void)hipEventDestroy(r.start);
        (void)hipEventDestroy(r.stop);
      }
      S.pending.clear();
      S.plans.clear();
      S.host_plans.clear();
      N.plans.clear();
      for (auto& kv : N.devices) {  // the scratch arrays stay (static); what they hold is forgotten
        kv.second.resident = 0;
        kv.second.table.clear();
      }
      for (auto& kv : S.ws) {
        if (kv.second.ptr) (void)hipFree(kv.second.ptr);
        if (kv.second.last_use) (void)hipEventDestroy(kv.second.last_use);
      }
      S.ws.clear();
      for (auto& kv : S.event_pool)
        for (hipEvent_t e : kv.second) (void)hipEventDestroy(e);
      S.event_pool.clear();
      S.timing = false;
      S.totals = costa_timing{};
    }
    // outside the state lock: a ScaLAPACK-style call takes the layout cache's
    // lock and then the state lock, never the other way round
    release_scalapack_layouts();
    return COSTA_SUCCESS;
  });
}
