// Host side of liborth: argument validation, planning of the batched
// launches, workspace layout, descriptor upload and the C ABI of
// include/orth.h.  Every entry point validates everything before it
// enqueues anything; the library allocates no device memory.
#include <algorithm>
#include <array>
#include <atomic>
#include <climits>
#include <cstdarg>
#include <cstdlib>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <list>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"
#include "tile_order.h"

namespace orth {

// ------------------------------------------------------------ errors ----
static thread_local std::string g_last_error;

static int fail(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}
int report_error(int code, const char* msg) { return fail(code, msg); }
#define ORTH_HIP(call)                                                                  \
  do {                                                                                  \
    hipError_t e_ = (call);                                                             \
    if (e_ != hipSuccess) return fail(ORTH_EHIP, std::string(#call) + ": " + hipGetErrorString(e_)); \
  } while (0)

// ------------------------------------------------------ diagnostics ----
// Two environment switches, read once per process:
//   ORTH_LOG=1        every entry point prints its plan to stderr (matrices
//                     per bucket, work-table sizes, workspace layout);
//   ORTH_LOG=2        also every kernel launch (name and stream);
//   ORTH_DEBUG_SYNC=1 every kernel launch is followed by a synchronization
//                     of its stream, and a failing launch or kernel is
//                     printed with its name (the call still returns the
//                     error at its next HIP check).
static int env_level(const char* name) {
  const char* v = std::getenv(name);
  return v && *v ? std::atoi(v) : 0;
}
int log_level() {
  static const int lvl = env_level("ORTH_LOG");
  return lvl;
}
static bool debug_sync() {
  static const bool on = env_level("ORTH_DEBUG_SYNC") > 0;
  return on;
}
void log_line(const char* fmt, ...) {
  char buf[1024];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  std::fprintf(stderr, "[orth] %s\n", buf);
}

// ------------------------------------------------------------ timing ----
namespace {
struct TimingRec {
  std::string name;
  hipStream_t stream;   // the launch's stream: its end event pairs with the start on the same stream
  hipEvent_t a, b;
};
std::mutex g_tmu;
std::atomic<bool> g_timing{false};
std::vector<TimingRec> g_pending;
std::vector<hipEvent_t> g_event_pool;
std::map<std::string, std::pair<double, int64_t>> g_totals;
// per name, each launch's [start, end] in ms after the reference event (the
// first start drained since the last reset; kept out of the pool until then)
std::map<std::string, std::vector<std::pair<double, double>>> g_spans;
hipEvent_t g_ref = nullptr;
std::vector<std::string> g_filter;   // name prefixes of the launches to time (empty: all)

bool timed_locked(const char* name) {
  if (g_filter.empty()) return true;
  for (const auto& p : g_filter)
    if (std::strncmp(name, p.c_str(), p.size()) == 0) return true;
  return false;
}

std::vector<std::string> split_prefixes(const char* prefixes) {
  std::vector<std::string> out;
  if (!prefixes) return out;
  for (const char* p = prefixes;;) {
    const char* q = std::strchr(p, ';');
    const std::string one = q ? std::string(p, q) : std::string(p);
    if (!one.empty()) out.push_back(one);
    if (!q) break;
    p = q + 1;
  }
  return out;
}

hipEvent_t pool_event() {
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// the first failure of the last drain (for the error message)
std::string g_drain_err;

int drain_timing_locked() {
  int rc = ORTH_OK;
  g_drain_err.clear();
  auto failed = [&](const char* what, const std::string& name, hipError_t e) {
    if (rc == ORTH_OK) g_drain_err = std::string(what) + " of " + name + ": " + hipGetErrorString(e);
    rc = ORTH_EHIP;
  };
  for (auto& r : g_pending) {
    float ms = 0.f, at = 0.f;
    hipError_t e = r.a && r.b ? hipEventSynchronize(r.b) : hipErrorInvalidValue;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e == hipSuccess) {
      auto& t = g_totals[r.name];
      t.first += ms;
      t.second += 1;
      // events of every stream share the device's clock; a launch on
      // another stream may start before the reference event
      if (!g_ref) g_ref = r.a;
      e = hipEventElapsedTime(&at, g_ref, r.a);
      if (e != hipSuccess && hipEventElapsedTime(&at, r.a, g_ref) == hipSuccess) {
        at = -at;
        e = hipSuccess;
      }
      if (e == hipSuccess)
        g_spans[r.name].push_back({(double)at, (double)at + ms});
      else
        failed("start relative to the reference event", r.name, e);
    } else {
      failed("launch events", r.name, e);
    }
    if (r.a && r.a != g_ref) g_event_pool.push_back(r.a);
    if (r.b) g_event_pool.push_back(r.b);
  }
  g_pending.clear();
  return rc;
}

int drain_failed(int rc) { return fail(rc, ("timing events: " + g_drain_err).c_str()); }
}  // namespace

void timing_begin(const char* name, hipStream_t s) {
  if (log_level() >= 2) log_line("launch %s on stream %p", name, (void*)s);
  if (!g_timing) return;
  std::lock_guard<std::mutex> lk(g_tmu);
  if (!timed_locked(name)) return;
  TimingRec r{name, s, pool_event(), nullptr};
  // a failed record leaves the pair incomplete, which the read reports
  if (r.a && hipEventRecord(r.a, s) != hipSuccess) {
    g_event_pool.push_back(r.a);
    r.a = nullptr;
  }
  g_pending.push_back(r);
}

void timing_end(const char* name, hipStream_t s) {
  if (debug_sync()) {
    hipError_t e = hipPeekAtLastError();
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess)
      log_line("ORTH_DEBUG_SYNC: %s failed: %s", name, hipGetErrorString(e));
    else if (log_level() >= 2)
      log_line("ORTH_DEBUG_SYNC: %s done", name);
  }
  if (!g_timing) return;
  std::lock_guard<std::mutex> lk(g_tmu);
  if (!timed_locked(name)) return;
  for (auto it = g_pending.rbegin(); it != g_pending.rend(); ++it) {
    if (it->b == nullptr && it->stream == s && it->name == name) {
      it->b = pool_event();
      if (it->b && hipEventRecord(it->b, s) != hipSuccess) {
        g_event_pool.push_back(it->b);
        it->b = nullptr;
      }
      break;
    }
  }
}

// ------------------------------------------------------- side streams ----
// Independent parts of one call (the small-matrix kernels beside the tiled
// path) run on side streams.  They fork from the caller's stream once the
// call's tables are uploaded (an event recorded there, waited on by each
// side stream) and join back (an event per side stream, waited on by the
// caller's stream) before anything that reads their results, so the
// caller sees one stream.  Side streams have the default priority.  Every
// host thread keeps its own per device, so the records and waits of one
// call are issued in order by one thread; they live until the process ends.
namespace {
constexpr int kSides = 2;
struct SideSet {
  hipStream_t st[kSides] = {};
  hipEvent_t fork = nullptr;
  hipEvent_t join[kSides] = {};
};

// The side set of the device that runs the caller's stream `s` (created
// with that device current, which is restored afterwards).
hipError_t side_set(hipStream_t s, SideSet** out) {
  thread_local std::map<int, SideSet> sets;
  hipDevice_t dev = 0;
  hipError_t e = hipStreamGetDevice(s, &dev);
  if (e != hipSuccess) return e;
  SideSet& S = sets[dev];
  if (!S.fork) {
    int cur = 0;
    e = hipGetDevice(&cur);
    if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
    if (e != hipSuccess) return e;
    SideSet n;
    for (int i = 0; i < kSides && e == hipSuccess; ++i) e = hipStreamCreateWithFlags(&n.st[i], hipStreamNonBlocking);
    for (int i = 0; i < kSides && e == hipSuccess; ++i)
      e = hipEventCreateWithFlags(&n.join[i], hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&n.fork, hipEventDisableTiming);
    if (cur != dev) {
      const hipError_t r = hipSetDevice(cur);
      if (e == hipSuccess) e = r;
    }
    if (e != hipSuccess) return e;
    S = n;
  }
  *out = &S;
  return hipSuccess;
}

// The fork and join of one call.  side(i) is the caller's stream until
// fork() has succeeded; a fork that an error path leaves open is joined by
// the destructor, so no side work outlives the caller's view of the call.
class Fork {
 public:
  explicit Fork(hipStream_t s) : s_(s) {}
  Fork(const Fork&) = delete;
  Fork& operator=(const Fork&) = delete;
  ~Fork() {
    if (forked_) (void)join();
  }
  hipError_t fork() {
    hipError_t e = side_set(s_, &S_);
    if (e == hipSuccess) e = hipEventRecord(S_->fork, s_);
    for (int i = 0; i < kSides && e == hipSuccess; ++i) e = hipStreamWaitEvent(S_->st[i], S_->fork, 0);
    forked_ = e == hipSuccess;
    return e;
  }
  hipStream_t side(int i) const { return forked_ ? S_->st[i] : s_; }
  hipError_t join() {
    if (!forked_) return hipSuccess;
    forked_ = false;
    hipError_t first = hipSuccess;
    for (int i = 0; i < kSides; ++i) {
      hipError_t e = hipEventRecord(S_->join[i], S_->st[i]);
      if (e == hipSuccess) e = hipStreamWaitEvent(s_, S_->join[i], 0);
      if (first == hipSuccess) first = e;
    }
    return first;
  }

 private:
  hipStream_t s_;
  SideSet* S_ = nullptr;
  bool forked_ = false;
};
}  // namespace

// ------------------------------------------------- descriptor staging ----
// Descriptor tables are built on the host and copied into the caller's
// workspace (the regions that each call's layout reserves for them).  The
// copy source is a pinned staging buffer from a process-wide pool.  A
// buffer is taken only when the copy that last read it has completed
// (hipEventQuery, which does not block); when no idle buffer is large
// enough a new one is allocated (pinned host memory).  Buffers are never
// freed while the pool is below kStageMax buffers, so a call neither
// frees memory nor waits.  With kStageMax copies still in flight (that
// many calls enqueued ahead of the device), a call waits for the oldest
// one (and replaces its buffer if it is too small): the one point where
// the host blocks, documented at the boundary.
namespace {
struct StageSlot {
  void* buf = nullptr;
  size_t cap = 0;
  hipEvent_t done = nullptr;
  uint64_t seq = 0;          // order of last use (oldest = smallest)
};
constexpr size_t kStageMax = 64;
std::mutex g_smu;
std::vector<StageSlot> g_stage;
uint64_t g_stage_seq = 0;

bool slot_idle(const StageSlot& sl) { return !sl.done || hipEventQuery(sl.done) == hipSuccess; }
}  // namespace

// Host image of a call's tables: the spans that put() fills (workspace
// offset, bytes), their bytes back to back.  Only the spans are copied; a
// span that starts less than kSpanGap bytes after the previous one (in
// increasing offset order) extends it over the gap instead, which saves a
// copy call for a few zero bytes.
struct TableImage {
  static constexpr size_t kSpanGap = 64 << 10;
  std::vector<unsigned char> data;
  std::vector<std::pair<size_t, size_t>> spans;
  void add(size_t off, const void* p, size_t bytes) {
    if (!bytes) return;
    if (!spans.empty()) {
      const size_t end = spans.back().first + spans.back().second;
      if (off >= end && off - end < kSpanGap) {
        data.resize(data.size() + (off - end), 0);
        spans.back().second += off - end;
        const size_t at = data.size();
        data.resize(at + bytes);
        std::memcpy(data.data() + at, p, bytes);
        spans.back().second += bytes;
        return;
      }
    }
    const size_t at = data.size();
    data.resize(at + bytes);
    std::memcpy(data.data() + at, p, bytes);
    spans.push_back({off, bytes});
  }
};

static int upload_tables(const TableImage& img, void* dst, hipStream_t s) {
  if (img.data.empty()) return ORTH_OK;
  // a captured copy would read its staging buffer at replay, after later
  // calls have refilled it: calls with tables refuse a capturing stream
  // (this is their first enqueue, so nothing is left half-captured)
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  ORTH_HIP(hipStreamIsCapturing(s, &cap));
  if (cap != hipStreamCaptureStatusNone)
    return fail(ORTH_EUNSUPPORTED, "the call cannot be captured into a HIP graph: its descriptor tables are "
                                   "copied from staging buffers that later calls reuse");
  std::lock_guard<std::mutex> lk(g_smu);
  const size_t total = img.data.size();
  // the smallest idle buffer that fits
  StageSlot* sl = nullptr;
  for (auto& c : g_stage)
    if (c.cap >= total && (!sl || c.cap < sl->cap) && slot_idle(c)) sl = &c;
  if (!sl) {
    size_t cap = std::max<size_t>(total, 1 << 16);
    cap = (cap + 4095) & ~size_t(4095);
    if (g_stage.size() < kStageMax) {
      StageSlot n;
      ORTH_HIP(hipHostMalloc(&n.buf, cap, hipHostMallocDefault));
      n.cap = cap;
      const hipError_t e = hipEventCreateWithFlags(&n.done, hipEventDisableTiming);
      if (e != hipSuccess) {
        (void)hipHostFree(n.buf);
        return fail(ORTH_EHIP, std::string("hipEventCreateWithFlags: ") + hipGetErrorString(e));
      }
      g_stage.push_back(n);
      sl = &g_stage.back();
    } else {
      // every buffer is in flight: wait for the oldest copy
      sl = &*std::min_element(g_stage.begin(), g_stage.end(),
                              [](const StageSlot& a, const StageSlot& b) { return a.seq < b.seq; });
      ORTH_HIP(hipEventSynchronize(sl->done));
      if (sl->cap < total) {
        ORTH_HIP(hipHostFree(sl->buf));
        sl->buf = nullptr;
        sl->cap = 0;
        ORTH_HIP(hipHostMalloc(&sl->buf, cap, hipHostMallocDefault));
        sl->cap = cap;
      }
    }
  }
  sl->seq = ++g_stage_seq;
  std::memcpy(sl->buf, img.data.data(), total);
  size_t at = 0;
  for (const auto& sp : img.spans) {
    ORTH_HIP(hipMemcpyAsync(static_cast<unsigned char*>(dst) + sp.first, static_cast<unsigned char*>(sl->buf) + at,
                            sp.second, hipMemcpyHostToDevice, s));
    at += sp.second;
  }
  ORTH_HIP(hipEventRecord(sl->done, s));
  return ORTH_OK;
}

// ----------------------------------------------------------- plan cache ---
// The plans of recent calls, keyed by the exact argument values that
// determine them (descriptors, options, workspace address): a call that
// repeats an earlier one (a training loop) skips the host planning, which
// costs from tens of microseconds to tens of milliseconds.  The descriptor
// tables are still copied into the workspace on every call, so nothing
// depends on the workspace's contents between calls.  ORTH_PLAN_CACHE=0
// turns the cache off.
namespace {
struct PlanKey {
  std::string k;
  template <typename T>
  void add(const T& v) {
    k.append(reinterpret_cast<const char*>(&v), sizeof(T));
  }
  void add_bytes(const void* p, size_t n) {
    if (n) k.append(static_cast<const char*>(p), n);
  }
  void add_opts(const orth_bjorck_opts* o) {
    add(o->iters);
    add(o->beta);
    add(o->prescale);
    add(o->in_dtype);
    add(o->out_dtype);
    add(o->compute);
    add(o->power_iters);
    add(o->u);
    add(o->tile);
    add(o->saved);
  }
};

bool plan_cache_on() {
  static const bool on = [] {
    const char* v = std::getenv("ORTH_PLAN_CACHE");
    return !(v && *v && std::atoi(v) == 0);
  }();
  return on;
}

template <typename Plan>
class PlanCache {
 public:
  // build fills a plan; seal_plan(Plan&) seals its GEMM lists so that the
  // cached plan is never modified again
  template <typename Build>
  std::shared_ptr<const Plan> get(const std::string& key, Build&& build) {
    if (plan_cache_on()) {
      std::lock_guard<std::mutex> lk(mu_);
      for (auto it = lru_.begin(); it != lru_.end(); ++it)
        if (it->first == key) {
          lru_.splice(lru_.begin(), lru_, it);
          return lru_.front().second;
        }
    }
    auto p = std::make_shared<Plan>();
    build(*p);
    seal_plan(*p);
    if (plan_cache_on()) {
      std::lock_guard<std::mutex> lk(mu_);
      lru_.emplace_front(key, p);
      if (lru_.size() > kEntries) lru_.pop_back();
    }
    return p;
  }

 private:
  static constexpr size_t kEntries = 4;
  std::mutex mu_;
  std::list<std::pair<std::string, std::shared_ptr<const Plan>>> lru_;
};
}  // namespace

// ------------------------------------------------------------ layout ----
namespace {
constexpr size_t kAlign = 256;
inline size_t align_up(size_t v, size_t a = kAlign) { return (v + a - 1) / a * a; }
inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }
// Base address a plan is laid out from: the workspace, or (sizing only, or
// a missing workspace that the call then rejects) a stand-in that is never
// dereferenced, so that the planners' address arithmetic never starts from
// a null pointer.
inline unsigned char* plan_base(void* ws) {
  return ws ? static_cast<unsigned char*>(ws) : reinterpret_cast<unsigned char*>(uintptr_t(1) << 44);
}

struct Arena {
  size_t off = 0;
  size_t take(size_t bytes) {
    off = align_up(off);
    const size_t o = off;
    off += bytes;
    return o;
  }
};

// fp32 GEMM work of one launch: one item per product, one GemmTile per
// 64 x 64 output tile (consecutive tiles of a product share its item).  In
// the workspace: the items, then the tiles.
static_assert(sizeof(GemmItem) % 8 == 0 && sizeof(GemmItem) == 8 * 8 + 14 * 8 + 18 * 4,
              "GemmItem must have no padding: items are compared bytewise");
// Products added whole (add_all) get their tiles at finalize().  (128 x 128
// tiles for lists of large products were measured 5-30% slower with this
// kernel's register-staged loads, so every list uses 64 x 64.)
struct GemmList {
  std::vector<GemmItem> items;
  std::vector<GemmTile> tiles;
  std::vector<int32_t> pending;   // add_all products without tiles yet
  int64_t pending64 = 0;          // their tile count
  GemmItem last{};   // items.back() with its tile and mirror fields cleared
  int64_t n_km = 0;  // trailing tiles for the k-major instantiation (set by put)
  size_t size() const { return tiles.size() + (size_t)pending64; }
  void clear() {
    items.clear();
    tiles.clear();
    pending.clear();
    pending64 = 0;
    n_km = 0;
  }
  // single-pair products with both operands stored k-major
  static bool kmajor(const GemmItem& it) { return it.a_trans && it.b_trans && it.K2 <= 0 && it.pair_count == 0; }
  // moves the k-major tiles to the end (stable: each part keeps its order)
  void partition_km() {
    auto it = std::stable_partition(tiles.begin(), tiles.end(),
                                    [&](const GemmTile& t) { return !kmajor(items[t.item]); });
    n_km = tiles.end() - it;
  }
  void finalize() {
    for (int32_t idx : pending)
      for (int a = 0; a < (items[idx].M + 63) / 64; ++a)
        for (int b = 0; b < (items[idx].N + 63) / 64; ++b) tiles.push_back(GemmTile{idx, a, b, 0});
    pending.clear();
    pending64 = 0;
  }
  // one tile, given as a whole item with its ti, tj (and mirror for an
  // off-diagonal tile); it shares the previous tile's item when the rest
  // matches
  void push_back(const GemmItem& g) {
    GemmItem k = g;
    k.ti = k.tj = 0;
    k.mirror = 0;
    if (items.empty() || std::memcmp(&k, &last, sizeof k) != 0) {
      items.push_back(k);
      last = k;
    }
    if (g.mirror) items.back().mirror = 1;
    tiles.push_back(GemmTile{(int32_t)items.size() - 1, g.ti, g.tj, 0});
  }
  // every tile of proto's M x N output (made by finalize)
  void add_all(const GemmItem& proto) {
    GemmItem k = proto;
    k.ti = k.tj = 0;
    items.push_back(k);
    last = k;
    last.mirror = 0;
    pending.push_back((int32_t)items.size() - 1);
    pending64 += (int64_t)((proto.M + 63) / 64) * ((proto.N + 63) / 64);
  }
  size_t items_bytes() const { return align_up(items.size() * sizeof(GemmItem)); }
  // workspace bytes for at most n tiles, each of its own product
  static size_t bound(size_t n) { return align_up(n * sizeof(GemmItem)) + align_up(n * sizeof(GemmTile)); }
  size_t bytes() const { return items_bytes() + align_up(tiles.size() * sizeof(GemmTile)); }
};

// Tiles of the products added whole, and the k-major tiles moved to the
// end: a list is sealed once its plan is complete, before any upload.
void seal(GemmList& g) {
  g.finalize();
  g.partition_km();
}
void put(TableImage& img, size_t off, const GemmList& g) {
  img.add(off, g.items.data(), g.items.size() * sizeof(GemmItem));
  img.add(off + g.items_bytes(), g.tiles.data(), g.tiles.size() * sizeof(GemmTile));
}
void put(TableImage& img, size_t off, GemmList& g) {
  seal(g);
  put(img, off, static_cast<const GemmList&>(g));
}

// Longest reductions first (stable: a product's tiles keep their order), so
// that short tiles fill a launch's tail; extra pairs are counted at the
// first pair's depth.
void longest_first(GemmList& g) {
  g.finalize();
  auto work = [&](const GemmTile& t) {
    const GemmItem& it = g.items[t.item];
    return (int64_t)it.K * (1 + it.pair_count) + it.K2;
  };
  std::stable_sort(g.tiles.begin(), g.tiles.end(),
                   [&](const GemmTile& a, const GemmTile& b) { return work(a) > work(b); });
}

hipError_t launch_list(const unsigned char* ws, size_t off, const GemmList& g, const char* name, hipStream_t s,
                       int step = 0, const GemmPair* pairs = nullptr) {
  return launch_gemm_f32(reinterpret_cast<const GemmItem*>(ws + off),
                         reinterpret_cast<const GemmTile*>(ws + off + g.items_bytes()), (int)g.size(), name, s,
                         step, pairs, (int)g.n_km);
}

}  // namespace

// ---------------------------------------------------- orthogonalize plan --
namespace {
enum Bucket { SMALL32 = 0, SMALL64 = 1, TILED_F32 = 2, TILED_BF16_128 = 3, TILED_BF16_256 = 4 };

struct MatPlan {
  int bucket;
  int32_t M, N, Mp, Np, transposed;
};

// bf16 tile tables of one size class: the Gram and the update tiles of all
// its matrices, for both ping-pong parities (step t uses parity t & 1).
enum { TAB_GRAM = 0, TAB_UPDATE = 2, N_TABS = 4 };  // + parity

struct OrthoPlan {
  std::vector<MatPlan> mp;
  std::vector<SmallMat> small[2];
  std::vector<TiledMat> tiled;                  // host copy with device pointers
  std::vector<TileItem> partial_items, scale_items, writeout_items;
  std::vector<TileItem> tabs[2][N_TABS];        // bf16: [0] = 128 tiles, [1] = 256 tiles
  GemmList f32_gram, f32_update[2];
  std::vector<PowerItem> power[2];              // spectral: v -> x and x -> y products
  int max_mp[2] = {32, 32};
  int total_partials = 0;
  // offsets in the workspace
  size_t off_small[2] = {0, 0}, off_tiled = 0, off_partial_items = 0, off_scale_items = 0, off_writeout_items = 0;
  size_t off_tabs[2][N_TABS] = {};
  size_t off_f32_gram = 0, off_f32_update[2] = {0, 0};
  size_t off_power[2] = {0, 0};
  size_t off_partials = 0, off_inv = 0, off_status = 0;
  size_t table_bytes = 0, total_bytes = 0;
  int n_out_iter = 0;   // tiled matrices whose output buffer holds the fp32 iterate
};

// ORTH_LOG plan dump of an orthogonalization call
void log_ortho_plan(const char* entry, const OrthoPlan& P, const orth_bjorck_opts* o) {
  if (log_level() < 1) return;
  int cnt[5] = {0, 0, 0, 0, 0};
  for (const auto& q : P.mp) ++cnt[q.bucket];
  log_line("%s: %zu matrices (fused small N<=32: %d, N<=64: %d; tiled fp32: %d; bf16 128-tiles: %d, 256-tiles: %d), "
           "T=%d beta=%g prescale=%d compute=%s",
           entry, P.mp.size(), cnt[SMALL32], cnt[SMALL64], cnt[TILED_F32], cnt[TILED_BF16_128], cnt[TILED_BF16_256],
           o->iters, o->beta, o->prescale, o->compute == ORTH_COMPUTE_BF16 ? "bf16" : "f32");
  for (int cls = 0; cls < 2; ++cls)
    if (!P.tabs[cls][TAB_GRAM].empty())
      log_line("%s: bf16 %d-tiles per step: %zu Gram + %zu update", entry, cls ? 256 : 128,
               P.tabs[cls][TAB_GRAM].size(), P.tabs[cls][TAB_UPDATE].size());
  if (P.f32_gram.size())
    log_line("%s: fp32 64-tiles per step: %zu Gram + %zu update", entry, P.f32_gram.size(), P.f32_update[0].size());
  log_line("%s: workspace %zu bytes (tables %zu); outputs holding the fp32 iterate: %d", entry, P.total_bytes,
           P.table_bytes, P.n_out_iter);
  if (log_level() >= 3)
    for (size_t i = 0; i < P.mp.size(); ++i)
      log_line("%s:   matrix %zu: %d x %d (tall), padded %d x %d, bucket %d%s", entry, i, P.mp[i].M, P.mp[i].N,
               P.mp[i].Mp, P.mp[i].Np, P.mp[i].bucket, P.mp[i].transposed ? ", transposed" : "");
}

void seal_plan(OrthoPlan& P) {
  seal(P.f32_gram);
  seal(P.f32_update[0]);
  seal(P.f32_update[1]);
}

int validate_ortho(const orth_mat* mats, int32_t n, const orth_bjorck_opts* o) {
  if (n < 0) return fail(ORTH_EINVAL, "n must be >= 0");
  if (n > 0 && !mats) return fail(ORTH_EINVAL, "mats is NULL");
  if (!o) return fail(ORTH_EINVAL, "opts is NULL");
  if (o->iters < 0) return fail(ORTH_EINVAL, "iters must be >= 0");
  if (!(o->beta > 0.f && o->beta <= 0.5f)) return fail(ORTH_EINVAL, "beta must lie in (0, 0.5]");
  if (o->prescale != ORTH_PRESCALE_NONE && o->prescale != ORTH_PRESCALE_FROBENIUS &&
      o->prescale != ORTH_PRESCALE_SPECTRAL)
    return fail(ORTH_EINVAL, "unknown prescale mode");
  if (o->prescale == ORTH_PRESCALE_SPECTRAL) {
    if (o->power_iters < 1 || o->power_iters > 1024) return fail(ORTH_EINVAL, "power_iters must lie in [1, 1024]");
    if (n > 0 && !o->u) return fail(ORTH_EINVAL, "spectral pre-scaling needs the cached vectors u");
  }
  if ((o->in_dtype != ORTH_F32 && o->in_dtype != ORTH_BF16) || (o->out_dtype != ORTH_F32 && o->out_dtype != ORTH_BF16))
    return fail(ORTH_EINVAL, "unknown dtype");
  if (o->compute != ORTH_COMPUTE_F32 && o->compute != ORTH_COMPUTE_BF16) return fail(ORTH_EINVAL, "unknown compute mode");
  if (o->tile != 0 && o->tile != 128 && o->tile != 256) return fail(ORTH_EINVAL, "tile must be 0, 128 or 256");
  for (int i = 0; i < n; ++i) {
    const orth_mat& m = mats[i];
    char buf[160];
    if (!m.in || !m.out) {
      snprintf(buf, sizeof buf, "matrix %d: NULL data pointer", i);
      return fail(ORTH_EINVAL, buf);
    }
    if (m.rows < 1 || m.cols < 1 || m.rows > (1 << 20) || m.cols > (1 << 20)) {
      snprintf(buf, sizeof buf, "matrix %d: rows and cols must be in [1, 2^20]", i);
      return fail(ORTH_EINVAL, buf);
    }
    if (m.ld_in < m.cols || m.ld_out < m.cols) {
      snprintf(buf, sizeof buf, "matrix %d: leading dimension smaller than cols", i);
      return fail(ORTH_EINVAL, buf);
    }
    if (m.in == m.out && (o->in_dtype != o->out_dtype || m.ld_in != m.ld_out)) {
      snprintf(buf, sizeof buf, "matrix %d: in-place needs equal dtypes and leading dims", i);
      return fail(ORTH_EINVAL, buf);
    }
  }
  return ORTH_OK;
}

// Builds the whole plan; device pointers are derived from `ws` (may be
// nullptr when only sizing).
void build_ortho_plan(const orth_mat* mats, int32_t n, const orth_bjorck_opts* o, OrthoPlan& P,
                      unsigned char* ws, bool want_status_scratch) {
  const bool bf16 = o->compute == ORTH_COMPUTE_BF16;
  P.mp.resize(n);
  std::vector<int> tiled_of(n, -1);
  int n_tiled = 0;
  std::vector<std::pair<int, int>> dims(n);
  for (int i = 0; i < n; ++i)
    dims[i] = {std::max(mats[i].rows, mats[i].cols), std::min(mats[i].rows, mats[i].cols)};
  const bool big_tiles = use_big_tiles(dims, o->tile);
  for (int i = 0; i < n; ++i) {
    const orth_mat& m = mats[i];
    MatPlan& q = P.mp[i];
    q.transposed = m.rows < m.cols;
    q.M = std::max(m.rows, m.cols);
    q.N = std::min(m.rows, m.cols);
    if (q.N <= 64 && q.M <= 128) {
      q.bucket = q.N <= 32 ? SMALL32 : SMALL64;
      q.Mp = (int32_t)round_up(q.M, 32);
      q.Np = q.N <= 32 ? 32 : 64;
    } else if (!bf16) {
      q.bucket = TILED_F32;
      q.Mp = (int32_t)round_up(q.M, 64);
      q.Np = (int32_t)round_up(q.N, 64);
    } else if (q.N >= 1024 && big_tiles) {
      q.bucket = TILED_BF16_256;
      q.Mp = (int32_t)round_up(q.M, 256);
      q.Np = (int32_t)round_up(q.N, 256);
    } else {
      q.bucket = TILED_BF16_128;
      q.Mp = (int32_t)round_up(q.M, 128);
      q.Np = (int32_t)round_up(q.N, 128);
    }
    if (q.bucket >= TILED_F32) tiled_of[i] = n_tiled++;
  }

  // bf16 tile tables (matrix indices only; no device pointers needed)
  for (int cls = 0; cls < 2; ++cls) {
    const int bucket = cls ? TILED_BF16_256 : TILED_BF16_128;
    const int tsz = cls ? 256 : 128;
    std::vector<int> members;
    for (int i = 0; i < n; ++i)
      if (P.mp[i].bucket == bucket) members.push_back(i);
    std::vector<TileItem> g[2], u[2];
    // longest tiles first (a Gram tile runs over Mp, an update tile over Np),
    // so that the short ones fill the launch's tail
    std::vector<int> gm = members, um = members;
    std::stable_sort(gm.begin(), gm.end(), [&](int a, int b) { return P.mp[a].Mp > P.mp[b].Mp; });
    std::stable_sort(um.begin(), um.end(), [&](int a, int b) { return P.mp[a].Np > P.mp[b].Np; });
    std::vector<std::pair<int, int>> gram_mats;
    for (int i : gm) gram_mats.push_back({tiled_of[i], P.mp[i].Np / tsz});
    const std::vector<TileItem> gt = bf16_gram_tiles(gram_mats);
    std::vector<TileItem> ut;
    for (int i : um) bf16_update_tiles(tiled_of[i], P.mp[i].Mp / tsz, P.mp[i].Np / tsz, ut);
    for (int par = 0; par < 2; ++par) {
      for (TileItem t : gt) {
        t.flags = par ? TILE_PARITY : 0;
        g[par].push_back(t);
      }
      for (TileItem t : ut) {
        t.flags = TILE_UPDATE | (par ? TILE_PARITY : 0);
        u[par].push_back(t);
      }
    }
    // dispatched in the order bf16_matrix_tiles builds (tile_order.h)
    for (int par = 0; par < 2; ++par) {
      P.tabs[cls][TAB_GRAM + par] = g[par];
      P.tabs[cls][TAB_UPDATE + par] = u[par];
    }
  }

  // table region
  Arena A;
  int n_small[2] = {0, 0};
  for (auto& q : P.mp)
    if (q.bucket <= SMALL64) ++n_small[q.bucket];
  P.off_small[0] = A.take(sizeof(SmallMat) * n_small[0]);
  P.off_small[1] = A.take(sizeof(SmallMat) * n_small[1]);
  P.off_tiled = A.take(sizeof(TiledMat) * n_tiled);
  int64_t n_part = 0, n_scale = 0, n_fg = 0, n_fu = 0;
  for (int i = 0; i < n; ++i) {
    const MatPlan& q = P.mp[i];
    if (q.bucket <= SMALL64) continue;
    n_part += (int64_t)((mats[i].rows + 63) / 64) * ((mats[i].cols + 63) / 64);
    n_scale += (int64_t)(q.Mp / 64) * (q.Np / 64);
    if (q.bucket == TILED_F32) {
      const int64_t tn = q.Np / 64, tm = q.Mp / 64;
      n_fg += tn * (tn + 1) / 2;
      n_fu += tm * tn;
    }
  }
  P.off_partial_items = A.take(sizeof(TileItem) * n_part);
  P.off_scale_items = A.take(sizeof(TileItem) * n_scale);
  P.off_writeout_items = A.take(sizeof(TileItem) * n_part);
  for (int cls = 0; cls < 2; ++cls)
    for (int t = 0; t < N_TABS; ++t) P.off_tabs[cls][t] = A.take(sizeof(TileItem) * P.tabs[cls][t].size());
  P.off_f32_gram = A.take(GemmList::bound(n_fg));
  P.off_f32_update[0] = A.take(GemmList::bound(n_fu));
  P.off_f32_update[1] = A.take(GemmList::bound(n_fu));
  const bool spectral = o->prescale == ORTH_PRESCALE_SPECTRAL;
  int64_t n_pw[2] = {0, 0};
  if (spectral)
    for (int i = 0; i < n; ++i) {
      if (P.mp[i].bucket <= SMALL64) continue;
      n_pw[0] += (P.mp[i].M + 63) / 64;   // outputs of X v
      n_pw[1] += (P.mp[i].N + 63) / 64;   // outputs of X^T x
    }
  P.off_power[0] = A.take(sizeof(PowerItem) * n_pw[0]);
  P.off_power[1] = A.take(sizeof(PowerItem) * n_pw[1]);
  P.table_bytes = align_up(A.off);
  P.off_partials = A.take(sizeof(double) * n_part);
  P.off_inv = A.take(sizeof(float) * n_tiled);
  P.off_status = A.take(want_status_scratch ? sizeof(int32_t) * n : 0);

  auto dev = [&](size_t off) -> unsigned char* { return ws ? ws + off : nullptr; };

  // per-matrix buffers and descriptors
  int part_base = 0;
  int64_t u_off = 0;   // this matrix's cached vector in the packed array
  for (int i = 0; i < n; ++i) {
    const orth_mat& m = mats[i];
    const MatPlan& q = P.mp[i];
    float* u_i = spectral ? o->u + u_off : nullptr;
    u_off += q.N;
    if (q.bucket <= SMALL64) {
      SmallMat s{};
      s.u = u_i;
      s.in = m.in;
      s.out = m.out;
      s.ld_in = m.ld_in;
      s.ld_out = m.ld_out;
      s.rows = m.rows;
      s.cols = m.cols;
      s.M = q.M;
      s.N = q.N;
      s.Mp = q.Mp;
      s.transposed = q.transposed;
      s.status_index = i;
      P.small[q.bucket].push_back(s);
      P.max_mp[q.bucket] = std::max(P.max_mp[q.bucket], q.Mp);
      continue;
    }
    const int tiled_idx = tiled_of[i];
    TiledMat t{};
    t.in = m.in;
    t.out = m.out;
    t.ld_in = m.ld_in;
    t.ld_out = m.ld_out;
    t.rows = m.rows;
    t.cols = m.cols;
    t.M = q.M;
    t.N = q.N;
    t.Mp = q.Mp;
    t.Np = q.Np;
    t.transposed = q.transposed;
    t.status_index = i;
    const int pr = (m.rows + 63) / 64, pc = (m.cols + 63) / 64;
    t.partial_base = part_base;
    t.n_partials = pr * pc;
    part_base += pr * pc;
    const size_t elems = (size_t)q.Mp * q.Np;
    const size_t csz = bf16 ? 2 : 4;
    // An fp32 output with the iterate's own layout (tall, no padding, row
    // stride Np, 16-byte aligned) serves as the fp32 buffer that the last
    // step writes (bf16 products update their single buffer in place; fp32
    // ones alternate two, X_T landing in slot T mod 2): no workspace for it
    // and no write-out pass.  The pre-scaling reads the input in full
    // before anything is written there, so in-place calls qualify too.
    const bool out_iter = o->out_dtype == ORTH_F32 && !q.transposed && q.Mp == m.rows && q.Np == m.cols &&
                          m.ld_out == q.Np && (reinterpret_cast<uintptr_t>(m.out) & 15) == 0;
    const int last = bf16 ? 0 : (o->iters & 1);
    for (int k = 0; k < (bf16 ? 1 : 2); ++k)
      t.master[k] = out_iter && k == last ? static_cast<float*>(m.out)
                                          : reinterpret_cast<float*>(dev(A.take(elems * 4)));
    if (bf16) t.master[1] = nullptr;
    P.n_out_iter += out_iter;
    t.xc[0] = bf16 ? dev(A.take(elems * 2)) : nullptr;
    t.xc[1] = bf16 ? dev(A.take(elems * 2)) : nullptr;
    t.xt = bf16 ? nullptr : dev(A.take(elems * csz));   // the bf16 Gram reads X itself
    t.e = dev(A.take((size_t)q.Np * q.Np * csz));
    t.inv_norm = reinterpret_cast<float*>(dev(P.off_inv)) + tiled_idx;
    if (spectral) {
      t.u = u_i;
      t.pv = reinterpret_cast<double*>(dev(A.take(sizeof(double) * q.N)));
      t.px = reinterpret_cast<double*>(dev(A.take(sizeof(double) * q.M)));
      t.py = reinterpret_cast<double*>(dev(A.take(sizeof(double) * q.N)));
      t.sig = reinterpret_cast<double*>(dev(A.take(sizeof(double))));
      // X v is a row product of W for a tall input and a column product for
      // a wide one; X^T x the other way round
      for (int b = 0; b < (q.M + 63) / 64; ++b) P.power[0].push_back(PowerItem{tiled_idx, b, q.transposed, 0});
      for (int b = 0; b < (q.N + 63) / 64; ++b) P.power[1].push_back(PowerItem{tiled_idx, b, !q.transposed, 1});
    }
    P.tiled.push_back(t);

    for (int a = 0; a < pr; ++a)
      for (int b = 0; b < pc; ++b) {
        P.partial_items.push_back(TileItem{tiled_idx, a, b, 0});
        if (!out_iter) P.writeout_items.push_back(TileItem{tiled_idx, a, b, 0});
      }
    for (int a = 0; a < q.Mp / 64; ++a)
      for (int b = 0; b < q.Np / 64; ++b) P.scale_items.push_back(TileItem{tiled_idx, a, b, 0});

    if (q.bucket == TILED_F32) {
      const int tn = q.Np / 64, tm = q.Mp / 64;
      std::vector<TileItem> gt, ut;
      grouped_tiles(tiled_idx, tn, tn, 4, true, gt);
      grouped_tiles(tiled_idx, tm, tn, 4, false, ut);
      for (auto& g : gt) {
        GemmItem gi{};
        gi.A = t.xt;
        gi.B = t.xt;
        gi.C = t.e;
        gi.lda = gi.ldb = q.Mp;
        gi.ldc = q.Np;
        gi.M = gi.N = q.Np;
        gi.K = q.Mp;
        gi.ti = g.ti;
        gi.tj = g.tj;
        gi.a_dtype = gi.b_dtype = ORTH_F32;
        gi.epi = EPI_GRAM_E;
        gi.mirror = g.ti != g.tj;
        P.f32_gram.push_back(gi);
      }
      for (int par = 0; par < 2; ++par)
        for (auto& u : ut) {
          GemmItem gi{};
          gi.A = t.master[par];
          gi.B = t.e;
          gi.C = t.master[par ^ 1];
          gi.src = t.master[par];
          gi.dst2 = static_cast<float*>(t.xt);
          gi.lda = q.Np;
          gi.ldb = q.Np;
          gi.ldc = q.Np;
          gi.ld_src = q.Np;
          gi.ld2 = q.Mp;
          gi.M = q.Mp;
          gi.N = q.Np;
          gi.K = q.Np;
          gi.ti = u.ti;
          gi.tj = u.tj;
          gi.a_dtype = gi.b_dtype = ORTH_F32;
          gi.epi = EPI_UPDATE;
          gi.beta = o->beta;
          P.f32_update[par].push_back(gi);
        }
    }
  }
  P.total_partials = part_base;
  P.total_bytes = align_up(A.off);

  // XCD-aware physical order of the fp32 GEMM work lists
  longest_first(P.f32_gram);
  longest_first(P.f32_update[0]);
  longest_first(P.f32_update[1]);
}

template <typename T>
void put(TableImage& img, size_t off, const std::vector<T>& v) {
  img.add(off, v.data(), sizeof(T) * v.size());
}


int check_workspace(void* ws, size_t have, size_t need) {
  if (need == 0) return ORTH_OK;
  if (!ws) return fail(ORTH_EWORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % kAlign) return fail(ORTH_EWORKSPACE, "workspace must be 256-byte aligned");
  if (have < need) {
    char buf[128];
    snprintf(buf, sizeof buf, "workspace too small: %zu bytes given, %zu needed", have, need);
    return fail(ORTH_EWORKSPACE, buf);
  }
  return ORTH_OK;
}
}  // namespace

// ------------------------------------------------------- conv planning ---
namespace {
int validate_geom(const orth_conv_geom* g) {
  if (!g) return fail(ORTH_EINVAL, "geometry is NULL");
  if (g->cin < 1 || g->cout < 1 || g->k < 1 || g->stride < 1 || g->dilation < 1 || g->groups < 1)
    return fail(ORTH_EINVAL, "all conv sizes must be >= 1");
  if (g->cin > (1 << 20) || g->cout > (1 << 20) || g->k > 64 || g->stride > 64 || g->dilation > 1024)
    return fail(ORTH_EINVAL, "conv sizes out of range");
  if (g->cin % g->groups || g->cout % g->groups) return fail(ORTH_EINVAL, "groups must divide cin and cout");
  if (g->k < g->stride) return fail(ORTH_EUNSUPPORTED, "kernel size must be >= stride");
  int a = g->stride, b = g->dilation;
  while (b) {
    const int t = a % b;
    a = b;
    b = t;
  }
  if (g->stride > 1 && a != 1) return fail(ORTH_EUNSUPPORTED, "stride > 1 needs gcd(stride, dilation) == 1");
  if (g->k > g->stride && g->cin / g->groups < 2)
    return fail(ORTH_EUNSUPPORTED, "BCOP blocks need at least 2 channels per group");
  return ORTH_OK;
}

struct ConvPlan {
  std::vector<ComposeGroup> groups;
  GemmList proj_items;
  std::vector<GemmList> phase_gemm;
  std::vector<std::vector<CombineItem>> phase_comb;
  std::vector<int64_t> phase_max_elems;
  int64_t init_max = 0, scatter_max = 0;
  std::vector<TapItem> scatter;                 // final taps -> OIHW kernel, per group
  size_t off_groups = 0, off_proj_items = 0, off_scatter = 0;
  std::vector<size_t> off_phase_gemm, off_phase_comb;
  size_t table_bytes = 0, total_bytes = 0;
};

void seal_plan(ConvPlan& P) {
  seal(P.proj_items);
  for (auto& g : P.phase_gemm) seal(g);
}

int validate_conv_descs(const orth_conv_desc* d, int32_t n, int32_t dtype) {
  if (n < 0) return fail(ORTH_EINVAL, "n must be >= 0");
  if (n > 0 && !d) return fail(ORTH_EINVAL, "descs is NULL");
  if (dtype != ORTH_F32 && dtype != ORTH_BF16) return fail(ORTH_EINVAL, "unknown dtype");
  for (int i = 0; i < n; ++i) {
    const int rc = validate_geom(&d[i].geom);
    if (rc) return rc;
    const int nproj = 2 * (d[i].geom.k - d[i].geom.stride);
    if (!d[i].rko || !d[i].kernel || (nproj > 0 && !d[i].proj)) return fail(ORTH_EINVAL, "NULL conv data pointer");
  }
  return ORTH_OK;
}

void build_conv_plan(const orth_conv_desc* d, int32_t n, int32_t dtype, ConvPlan& P, unsigned char* ws) {
  const size_t esz = dtype == ORTH_BF16 ? 2 : 4;
  int max_kp = 1;
  for (int i = 0; i < n; ++i) max_kp = std::max(max_kp, d[i].geom.k - d[i].geom.stride + 1);
  const int n_phase = 2 * (max_kp - 1);
  // count
  int n_groups = 0;
  for (int i = 0; i < n; ++i) n_groups += d[i].geom.groups;
  Arena A;
  P.off_groups = A.take(sizeof(ComposeGroup) * n_groups);

  auto dev = [&](size_t off) -> unsigned char* { return ws ? ws + off : nullptr; };
  // item lists (pointers filled after buffer layout, so lay out buffers in a
  // second arena that starts after the tables; sizes of tables are counted first)
  P.phase_gemm.assign(n_phase, {});
  P.phase_comb.assign(n_phase, {});
  P.phase_max_elems.assign(n_phase, 0);

  struct Tmp {
    int layer, group;
  };
  std::vector<Tmp> tmp;
  for (int i = 0; i < n; ++i)
    for (int g = 0; g < d[i].geom.groups; ++g) tmp.push_back(Tmp{i, g});

  // counts of items to size the table region
  size_t n_proj_items = 0;
  std::vector<size_t> n_pg(n_phase, 0), n_pc(n_phase, 0);
  for (auto& t : tmp) {
    const orth_conv_geom& g = d[t.layer].geom;
    const int c = g.cin / g.groups, og = g.cout / g.groups, s = g.stride, k = g.k, kp = k - s + 1;
    const int nproj = 2 * (kp - 1);
    const size_t ct = (c + 63) / 64, ot = (og + 63) / 64;
    n_proj_items += nproj * ct * ct;
    for (int ph = 0; ph < n_phase; ++ph) {
      const bool vert = ph >= max_kp - 1;
      const int j = vert ? ph - (max_kp - 1) : ph;
      if (j >= kp - 1) continue;
      const int in_h = vert ? s + j : s, in_w = vert ? k : s + j;
      n_pg[ph] += (size_t)in_h * in_w * ot * ct;
      n_pc[ph] += 1;
    }
  }
  P.off_proj_items = A.take(GemmList::bound(n_proj_items));
  P.off_phase_gemm.resize(n_phase);
  P.off_phase_comb.resize(n_phase);
  for (int ph = 0; ph < n_phase; ++ph) {
    P.off_phase_gemm[ph] = A.take(GemmList::bound(n_pg[ph]));
    P.off_phase_comb[ph] = A.take(sizeof(CombineItem) * n_pc[ph]);
  }
  P.off_scatter = A.take(sizeof(TapItem) * n_groups);
  P.table_bytes = align_up(A.off);

  for (auto& t : tmp) {
    const orth_conv_desc& L = d[t.layer];
    const orth_conv_geom& g = L.geom;
    const int c = g.cin / g.groups, og = g.cout / g.groups, s = g.stride, k = g.k, kp = k - s + 1;
    const int h = c / 2, nproj = 2 * (kp - 1);
    ComposeGroup G{};
    G.rko = static_cast<const unsigned char*>(L.rko) + (size_t)t.group * og * c * s * s * esz;
    G.proj = nproj ? static_cast<const unsigned char*>(L.proj) + (size_t)t.group * nproj * c * h * esz : nullptr;
    G.kernel = L.kernel;
    const size_t tapbytes = (size_t)k * k * og * c * sizeof(float);
    G.taps[0] = reinterpret_cast<float*>(dev(A.take(tapbytes)));
    G.taps[1] = kp > 1 ? reinterpret_cast<float*>(dev(A.take(tapbytes))) : nullptr;
    G.y = kp > 1 ? reinterpret_cast<float*>(dev(A.take(tapbytes))) : nullptr;
    G.p = nproj ? reinterpret_cast<float*>(dev(A.take((size_t)nproj * c * c * sizeof(float)))) : nullptr;
    G.cout_g = og;
    G.c = c;
    G.h = h;
    G.k = k;
    G.s = s;
    G.group = t.group;
    G.nproj = nproj;
    const int gidx = (int)P.groups.size();
    P.init_max = std::max<int64_t>(P.init_max, (int64_t)s * s * og * c);
    P.scatter_max = std::max<int64_t>(P.scatter_max, (int64_t)k * k * og * c);

    for (int j = 0; j < nproj; ++j) {
      GemmItem gi{};
      gi.A = static_cast<const unsigned char*>(G.proj) + (size_t)j * c * h * esz;
      gi.B = gi.A;
      gi.C = G.p + (size_t)j * c * c;
      gi.lda = gi.ldb = h;
      gi.ldc = c;
      gi.M = gi.N = c;
      gi.K = h;
      gi.a_dtype = gi.b_dtype = dtype;
      gi.epi = EPI_STORE;
      P.proj_items.add_all(gi);
    }
    int cur = 0;
    for (int ph = 0; ph < n_phase; ++ph) {
      const bool vert = ph >= max_kp - 1;
      const int j = vert ? ph - (max_kp - 1) : ph;
      if (j >= kp - 1) continue;
      const int in_h = vert ? s + j : s, in_w = vert ? k : s + j;
      const int pj = vert ? (kp - 1) + j : j;  // projector index: h blocks first
      const size_t tap = (size_t)og * c;
      for (int a = 0; a < in_h; ++a)
        for (int b = 0; b < in_w; ++b) {
          GemmItem gi{};
          gi.A = G.taps[cur] + (size_t)(a * k + b) * tap;
          gi.B = G.p + (size_t)pj * c * c;
          gi.C = G.y + (size_t)(a * k + b) * tap;
          gi.lda = c;
          gi.ldb = c;
          gi.ldc = c;
          gi.M = og;
          gi.N = c;
          gi.K = c;
          gi.a_dtype = gi.b_dtype = ORTH_F32;
          gi.epi = EPI_STORE;
          P.phase_gemm[ph].add_all(gi);
        }
      P.phase_comb[ph].push_back(CombineItem{gidx, vert ? 1 : 0, in_h, in_w, cur, 0});
      const int out_taps = (in_h + (vert ? 1 : 0)) * (in_w + (vert ? 0 : 1));
      P.phase_max_elems[ph] = std::max<int64_t>(P.phase_max_elems[ph], (int64_t)out_taps * og * c);
      cur ^= 1;
    }
    G.cur = cur;
    P.groups.push_back(G);
    // kernel[group * og + o][i][a][b] = taps[a k + b][o][i]: the group's
    // slice of the OIHW kernel is the [og c][k k] transpose of its final taps
    P.scatter.push_back(TapItem{G.taps[cur], nullptr,
                                static_cast<unsigned char*>(L.kernel) + (size_t)t.group * og * c * k * k * esz,
                                nullptr, og, c, k, k, 0, 0});
  }
  P.total_bytes = align_up(A.off);
  for (int ph = 0; ph < n_phase; ++ph) longest_first(P.phase_gemm[ph]);
}
}  // namespace

// ----------------------------------------------- composition VJP plan ---
// Per group: the forward taps T_q (input of block step q) are recomputed in
// compact grids and kept; the gradient G runs back through the steps with
// Z = G P_q, the adjoint combine (dT and D) and dP_q = sum T_q^T D; finally
// dV_q = (dP_q + dP_q^T) V_q and the RKO gradient is read off the s x s taps.
// Steps are aligned across groups as in the forward plan (horizontal blocks
// at global steps 0.., vertical ones after the longest horizontal run).
namespace {
struct ConvVjpPlan {
  GemmList proj_items, last_dp, dv_items;
  std::vector<GemmList> fwd_gemm, bwd_gemm;
  std::vector<std::vector<TapItem>> fwd_comb, bwd_comb;
  std::vector<TapItem> rko_taps, grad_taps, rko_grad;
  std::vector<int64_t> fwd_max, bwd_max;
  int64_t rko_max = 0, grad_max = 0;
  size_t off_proj = 0, off_last_dp = 0, off_dv = 0, off_rko_taps = 0, off_grad_taps = 0, off_rko_grad = 0;
  std::vector<size_t> off_fwd_gemm, off_bwd_gemm, off_fwd_comb, off_bwd_comb;
  // saving forward only: the last block step into a k x k grid (G[0]) and
  // its scatter to the OIHW kernel
  std::vector<GemmList> save_gemm;
  std::vector<std::vector<TapItem>> save_comb;
  std::vector<TapItem> save_scatter;
  std::vector<int64_t> save_max;
  int64_t scatter_max = 0;
  std::vector<size_t> off_save_gemm, off_save_comb;
  size_t off_save_scatter = 0;
  size_t table_bytes = 0, total_bytes = 0;
};

void seal_plan(ConvVjpPlan& P) {
  seal(P.proj_items);
  seal(P.last_dp);
  seal(P.dv_items);
  for (auto& g : P.fwd_gemm) seal(g);
  for (auto& g : P.bwd_gemm) seal(g);
  for (auto& g : P.save_gemm) seal(g);
}

int validate_conv_vjp_descs(const orth_conv_vjp_desc* d, int32_t n, int32_t dtype) {
  if (n < 0) return fail(ORTH_EINVAL, "n must be >= 0");
  if (n > 0 && !d) return fail(ORTH_EINVAL, "descs is NULL");
  if (dtype != ORTH_F32 && dtype != ORTH_BF16) return fail(ORTH_EINVAL, "unknown dtype");
  for (int i = 0; i < n; ++i) {
    const int rc = validate_geom(&d[i].geom);
    if (rc) return rc;
    const int nproj = 2 * (d[i].geom.k - d[i].geom.stride);
    if (!d[i].rko || !d[i].grad_kernel || !d[i].grad_rko || (nproj > 0 && (!d[i].proj || !d[i].grad_proj)))
      return fail(ORTH_EINVAL, "NULL conv data pointer");
  }
  return ORTH_OK;
}

// every tile of an M x N output for the fp32 tile GEMM
void gemm_tiles(const GemmItem& proto, GemmList& out) { out.add_all(proto); }

// kernels: the layers' kernel outputs for a saving forward (nullptr
// otherwise; the layout does not depend on it)
void build_conv_vjp_plan(const orth_conv_vjp_desc* d, int32_t n, int32_t dtype, ConvVjpPlan& P,
                         unsigned char* ws, const void* const* kernels = nullptr) {
  const size_t esz = dtype == ORTH_BF16 ? 2 : 4;
  int max_kp = 1;
  for (int i = 0; i < n; ++i) max_kp = std::max(max_kp, d[i].geom.k - d[i].geom.stride + 1);
  const int n_phase = 2 * (max_kp - 1);
  P.fwd_gemm.assign(n_phase, {});
  P.bwd_gemm.assign(n_phase, {});
  P.fwd_comb.assign(n_phase, {});
  P.bwd_comb.assign(n_phase, {});
  P.fwd_max.assign(n_phase, 0);
  P.bwd_max.assign(n_phase, 0);
  P.save_gemm.assign(n_phase, {});
  P.save_comb.assign(n_phase, {});
  P.save_max.assign(n_phase, 0);

  // Two passes: the first (ws == nullptr inside) only counts table entries;
  // buffers follow the tables, so table sizes must be known first.
  for (int pass = 0; pass < 2; ++pass) {
    Arena A;
    if (pass == 1) {
      P.off_proj = A.take(GemmList::bound(P.proj_items.size()));
      P.off_last_dp = A.take(GemmList::bound(P.last_dp.size()));
      P.off_dv = A.take(GemmList::bound(P.dv_items.size()));
      P.off_rko_taps = A.take(sizeof(TapItem) * P.rko_taps.size());
      P.off_grad_taps = A.take(sizeof(TapItem) * P.grad_taps.size());
      P.off_rko_grad = A.take(sizeof(TapItem) * P.rko_grad.size());
      P.off_fwd_gemm.resize(n_phase);
      P.off_bwd_gemm.resize(n_phase);
      P.off_fwd_comb.resize(n_phase);
      P.off_bwd_comb.resize(n_phase);
      P.off_save_gemm.resize(n_phase);
      P.off_save_comb.resize(n_phase);
      for (int ph = 0; ph < n_phase; ++ph) {
        P.off_fwd_gemm[ph] = A.take(GemmList::bound(P.fwd_gemm[ph].size()));
        P.off_bwd_gemm[ph] = A.take(GemmList::bound(P.bwd_gemm[ph].size()));
        P.off_fwd_comb[ph] = A.take(sizeof(TapItem) * P.fwd_comb[ph].size());
        P.off_bwd_comb[ph] = A.take(sizeof(TapItem) * P.bwd_comb[ph].size());
        P.off_save_gemm[ph] = A.take(GemmList::bound(P.save_gemm[ph].size()));
        P.off_save_comb[ph] = A.take(sizeof(TapItem) * P.save_comb[ph].size());
      }
      P.off_save_scatter = A.take(sizeof(TapItem) * P.save_scatter.size());
      P.table_bytes = align_up(A.off);
      P.proj_items.clear();
      P.last_dp.clear();
      P.dv_items.clear();
      P.rko_taps.clear();
      P.grad_taps.clear();
      P.rko_grad.clear();
      for (int ph = 0; ph < n_phase; ++ph) {
        P.fwd_gemm[ph].clear();
        P.bwd_gemm[ph].clear();
        P.fwd_comb[ph].clear();
        P.bwd_comb[ph].clear();
        P.save_gemm[ph].clear();
        P.save_comb[ph].clear();
      }
      P.save_scatter.clear();
    }
    // (pass 0 lays out from the stand-in base: its addresses are discarded)
    auto dev = [&](size_t off) -> unsigned char* { return (pass == 1 ? ws : plan_base(nullptr)) + off; };
    auto fbuf = [&](int64_t elems) { return reinterpret_cast<float*>(dev(A.take((size_t)elems * 4))); };

    for (int li = 0; li < n; ++li) {
      const orth_conv_vjp_desc& L = d[li];
      const orth_conv_geom& g = L.geom;
      const int c = g.cin / g.groups, og = g.cout / g.groups, s = g.stride, k = g.k, kp = k - s + 1;
      const int h = c / 2, nq = 2 * (kp - 1);
      const int64_t tap = (int64_t)og * c;
      auto in_grid = [&](int q, int& gh, int& gw, int& v) {
        v = q >= kp - 1;
        gh = v ? s + (q - (kp - 1)) : s;
        gw = v ? k : s + q;
      };
      auto gphase = [&](int q) { return q < kp - 1 ? q : (max_kp - 1) + (q - (kp - 1)); };
      for (int grp = 0; grp < g.groups; ++grp) {
        const unsigned char* rko = static_cast<const unsigned char*>(L.rko) + (size_t)grp * og * c * s * s * esz;
        const unsigned char* proj =
            nq ? static_cast<const unsigned char*>(L.proj) + (size_t)grp * nq * c * h * esz : nullptr;
        const unsigned char* gk =
            static_cast<const unsigned char*>(L.grad_kernel) + (size_t)grp * og * c * k * k * esz;
        unsigned char* grko = static_cast<unsigned char*>(L.grad_rko) + (size_t)grp * og * c * s * s * esz;
        unsigned char* gproj = nq ? static_cast<unsigned char*>(L.grad_proj) + (size_t)grp * nq * c * h * esz : nullptr;
        // buffers
        std::vector<float*> Ts(std::max(nq, 1));
        int64_t max_in = s * s;
        for (int q = 0; q < std::max(nq, 1); ++q) {
          int gh = s, gw = s, v = 0;
          if (nq) in_grid(q, gh, gw, v);
          Ts[q] = fbuf((int64_t)gh * gw * tap);
          max_in = std::max<int64_t>(max_in, (int64_t)gh * gw);
        }
        float* Y = nq > 1 ? fbuf(max_in * tap) : nullptr;
        float* G[2] = {fbuf((int64_t)k * k * tap), fbuf((int64_t)k * k * tap)};
        float* Z = nq ? fbuf((int64_t)k * k * tap) : nullptr;
        float* D = nq ? fbuf(max_in * tap) : nullptr;
        float* Pm = nq ? fbuf((int64_t)nq * c * c) : nullptr;
        float* dP = nq ? fbuf((int64_t)nq * c * c) : nullptr;

        // forward recomputation
        P.rko_taps.push_back(TapItem{rko, nullptr, Ts[0], nullptr, og, c, s, s, 0, 0});
        P.rko_max = std::max<int64_t>(P.rko_max, (int64_t)s * s * tap);
        for (int j = 0; j < nq; ++j) {
          GemmItem gi{};
          gi.A = proj + (size_t)j * c * h * esz;
          gi.B = gi.A;
          gi.C = Pm + (size_t)j * c * c;
          gi.lda = gi.ldb = h;
          gi.ldc = c;
          gi.M = gi.N = c;
          gi.K = h;
          gi.a_dtype = gi.b_dtype = dtype;
          gi.epi = EPI_STORE;
          gemm_tiles(gi, P.proj_items);
        }
        for (int q = 0; q + 1 < nq; ++q) {
          int gh, gw, v;
          in_grid(q, gh, gw, v);
          const int ph = gphase(q);
          GemmItem gi{};
          gi.A = Ts[q];
          gi.B = Pm + (size_t)q * c * c;
          gi.C = Y;
          gi.lda = gi.ldb = gi.ldc = c;
          gi.M = gh * gw * og;
          gi.N = c;
          gi.K = c;
          gi.epi = EPI_STORE;
          gemm_tiles(gi, P.fwd_gemm[ph]);
          P.fwd_comb[ph].push_back(TapItem{Ts[q], Y, Ts[q + 1], nullptr, og, c, gh, gw, v, 0});
          P.fwd_max[ph] = std::max<int64_t>(P.fwd_max[ph], (int64_t)(gh + v) * (gw + 1 - v) * tap);
        }
        // saving forward: the last block step into the k x k grid G[0],
        // then the grid (or, without blocks, the s x s RKO taps) to OIHW
        if (nq) {
          const int q = nq - 1;
          int gh, gw, v;
          in_grid(q, gh, gw, v);
          const int ph = gphase(q);
          GemmItem gi{};
          gi.A = Ts[q];
          gi.B = Pm + (size_t)q * c * c;
          gi.C = Y ? Y : G[1];
          gi.lda = gi.ldb = gi.ldc = c;
          gi.M = gh * gw * og;
          gi.N = c;
          gi.K = c;
          gi.epi = EPI_STORE;
          gemm_tiles(gi, P.save_gemm[ph]);
          P.save_comb[ph].push_back(TapItem{Ts[q], gi.C, G[0], nullptr, og, c, gh, gw, v, 0});
          P.save_max[ph] = std::max<int64_t>(P.save_max[ph], (int64_t)(gh + v) * (gw + 1 - v) * tap);
        }
        void* kslice = kernels ? static_cast<unsigned char*>(const_cast<void*>(kernels[li])) +
                                     (size_t)grp * og * c * k * k * esz
                               : nullptr;
        P.save_scatter.push_back(TapItem{nq ? G[0] : Ts[0], nullptr, kslice, nullptr, og, c, k, k, 0, 0});
        P.scatter_max = std::max<int64_t>(P.scatter_max, (int64_t)k * k * tap);
        // gradient, last step first
        int cur = 0;
        P.grad_taps.push_back(TapItem{gk, nullptr, G[0], nullptr, og, c, k, k, 0, 0});
        P.grad_max = std::max<int64_t>(P.grad_max, (int64_t)k * k * tap);
        for (int q = nq - 1; q >= 0; --q) {
          int gh, gw, v;
          in_grid(q, gh, gw, v);
          const int ph = gphase(q);
          GemmItem gi{};
          gi.A = G[cur];
          gi.B = Pm + (size_t)q * c * c;
          gi.C = Z;
          gi.lda = gi.ldb = gi.ldc = c;
          gi.M = (gh + v) * (gw + 1 - v) * og;
          gi.N = c;
          gi.K = c;
          gi.epi = EPI_STORE;
          gemm_tiles(gi, P.bwd_gemm[ph]);
          if (q + 1 < nq) {   // dP of the step above, whose D is still in place
            int h1, w1, v1;
            in_grid(q + 1, h1, w1, v1);
            GemmItem gd{};
            gd.A = Ts[q + 1];
            gd.B = D;
            gd.a_trans = gd.b_trans = 1;
            gd.lda = gd.ldb = c;
            gd.K = h1 * w1 * og;
            gd.M = gd.N = c;
            gd.C = dP + (size_t)(q + 1) * c * c;
            gd.ldc = c;
            gd.epi = EPI_STORE;
            gemm_tiles(gd, P.bwd_gemm[ph]);
          }
          P.bwd_comb[ph].push_back(TapItem{G[cur], Z, G[cur ^ 1], D, og, c, gh, gw, v, 0});
          P.bwd_max[ph] = std::max<int64_t>(P.bwd_max[ph], (int64_t)gh * gw * tap);
          cur ^= 1;
        }
        if (nq) {
          GemmItem gd{};
          gd.A = Ts[0];
          gd.B = D;
          gd.a_trans = gd.b_trans = 1;
          gd.lda = gd.ldb = c;
          gd.K = s * s * og;
          gd.M = gd.N = c;
          gd.C = dP;
          gd.ldc = c;
          gd.epi = EPI_STORE;
          gemm_tiles(gd, P.last_dp);
        }
        for (int j = 0; j < nq; ++j) {
          GemmItem gv{};
          gv.A = dP + (size_t)j * c * c;
          gv.lda = c;
          gv.B = proj + (size_t)j * c * h * esz;
          gv.b_trans = 1;
          gv.ldb = h;
          gv.K = c;
          gv.A2 = gv.A;
          gv.a2_trans = 1;
          gv.lda2 = c;
          gv.B2 = gv.B;
          gv.b2_trans = 1;
          gv.ldb2 = h;
          gv.K2 = c;
          gv.M = c;
          gv.N = h;
          gv.a_dtype = ORTH_F32;
          gv.b_dtype = dtype;
          gv.C = gproj + (size_t)j * c * h * esz;
          gv.ldc = h;
          gv.c_dtype = dtype;
          gv.epi = EPI_STORE;
          gemm_tiles(gv, P.dv_items);
        }
        P.rko_grad.push_back(TapItem{G[cur], nullptr, grko, nullptr, og, c, s, s, 0, 0});
      }
    }
    P.total_bytes = align_up(A.off);
  }
}
}  // namespace

// ------------------------------------------------------ exponentials ----
// Exponential map: per matrix A = W - W^T, the spectral-normalization
// kernels on A (power iteration from the caller's cached vector, lower bound
// ||A||_F / sqrt(C)), Ahat = A / sigma, then P_k = P_{k-1} Ahat / k and
// What += P_k on the tile GEMM (Ahat^T = -Ahat, so the products read Ahat
// row-major and negate), and What written out.
// Conv exponential: L = scale (K - K*) as k x k taps, E = centred I + L,
// then Q_j = (Q_{j-1} ⊛ L) / j tap by tap (each output tap sums the products
// of the Q_{j-1} taps and L taps that meet there; L_{r,t}^T = -L_{k-1-r,k-1-t}
// lets every product read row-major operands) with E += Q_j, and E
// scattered to OIHW.
namespace {
struct ExpPlan {
  std::vector<ExpItem> items;
  std::vector<TiledMat> mats;                 // exp map: views of A for the spectral kernels
  std::vector<TileItem> partial_items, writeout_items;
  std::vector<PowerItem> power[2];
  std::vector<GemmList> steps;   // per power k = 2..p (index k - 2)
  std::vector<GemmPair> pairs;                // conv: operand pairs of all steps
  std::vector<TapItem> scatter;               // conv: E taps -> OIHW
  int64_t max_elems = 0, max_init = 0, max_scatter = 0;
  size_t off_items = 0, off_mats = 0, off_partial = 0, off_writeout = 0, off_power[2] = {}, off_pairs = 0,
         off_scatter = 0, off_partials = 0, off_inv = 0, off_status = 0;
  std::vector<size_t> off_steps;
  size_t table_bytes = 0, total_bytes = 0;
};

int validate_exp(const orth_mat* mats, int32_t n, const orth_exp_opts* o) {
  if (n < 0) return fail(ORTH_EINVAL, "n must be >= 0");
  if (n > 0 && !mats) return fail(ORTH_EINVAL, "mats is NULL");
  if (!o) return fail(ORTH_EINVAL, "opts is NULL");
  if (o->terms < 1 || o->terms > 64) return fail(ORTH_EINVAL, "terms must lie in [1, 64]");
  if (o->power_iters < 1 || o->power_iters > 1024) return fail(ORTH_EINVAL, "power_iters must lie in [1, 1024]");
  if (n > 0 && !o->u) return fail(ORTH_EINVAL, "u is NULL");
  if ((o->in_dtype != ORTH_F32 && o->in_dtype != ORTH_BF16) || (o->out_dtype != ORTH_F32 && o->out_dtype != ORTH_BF16))
    return fail(ORTH_EINVAL, "unknown dtype");
  for (int i = 0; i < n; ++i) {
    const orth_mat& m = mats[i];
    char buf[160];
    if (!m.in || !m.out || m.rows != m.cols || m.rows < 1 || m.rows > (1 << 16) || m.ld_in < m.cols ||
        m.ld_out < m.cols) {
      snprintf(buf, sizeof buf, "matrix %d: needs non-NULL square C x C data, 1 <= C <= 65536, ld >= C", i);
      return fail(ORTH_EINVAL, buf);
    }
    if (m.in == m.out) {
      snprintf(buf, sizeof buf, "matrix %d: in and out must differ", i);
      return fail(ORTH_EINVAL, buf);
    }
  }
  return ORTH_OK;
}

void build_exp_plan(const orth_mat* mats, int32_t n, const orth_exp_opts* o, ExpPlan& P, unsigned char* ws) {
  const int p = o->terms;
  P.steps.assign(std::max(p - 1, 0), {});
  int64_t n_part = 0, n_pw = 0, n_gemm = 0;
  for (int i = 0; i < n; ++i) {
    const int64_t t = (mats[i].rows + 63) / 64;
    n_part += t * t;
    n_pw += t;
    n_gemm += t * t;
  }
  Arena A;
  P.off_items = A.take(sizeof(ExpItem) * n);
  P.off_mats = A.take(sizeof(TiledMat) * n);
  P.off_partial = A.take(sizeof(TileItem) * n_part);
  P.off_writeout = A.take(sizeof(TileItem) * n_part);
  P.off_power[0] = A.take(sizeof(PowerItem) * n_pw);
  P.off_power[1] = A.take(sizeof(PowerItem) * n_pw);
  P.off_steps.resize(P.steps.size());
  for (size_t k = 0; k < P.steps.size(); ++k) P.off_steps[k] = A.take(GemmList::bound(n_gemm));
  P.table_bytes = align_up(A.off);
  P.off_partials = A.take(sizeof(double) * n_part);
  P.off_inv = A.take(sizeof(float) * n);
  P.off_status = A.take(sizeof(int32_t) * n);
  auto dev = [&](size_t off) -> unsigned char* { return ws ? ws + off : nullptr; };
  auto fbuf = [&](int64_t elems) { return reinterpret_cast<float*>(dev(A.take((size_t)elems * 4))); };
  int64_t u_off = 0;
  int part_base = 0;
  for (int i = 0; i < n; ++i) {
    const orth_mat& m = mats[i];
    const int C = m.rows;
    const int64_t cc = (int64_t)C * C;
    float* a = fbuf(cc);
    float* ahat = fbuf(cc);
    float* pp[2] = {fbuf(cc), p > 2 ? fbuf(cc) : nullptr};
    float* acc = fbuf(cc);
    float* inv = reinterpret_cast<float*>(dev(P.off_inv)) + i;
    TiledMat t{};
    t.in = a;
    t.out = m.out;
    t.ld_in = C;
    t.ld_out = m.ld_out;
    t.rows = t.cols = t.M = t.N = t.Mp = t.Np = C;
    t.status_index = i;
    const int tiles = (C + 63) / 64;
    t.partial_base = part_base;
    t.n_partials = tiles * tiles;
    part_base += tiles * tiles;
    t.master[0] = acc;
    t.inv_norm = inv;
    t.u = o->u + u_off;
    u_off += C;
    t.pv = reinterpret_cast<double*>(dev(A.take(sizeof(double) * C)));
    t.px = reinterpret_cast<double*>(dev(A.take(sizeof(double) * C)));
    t.py = reinterpret_cast<double*>(dev(A.take(sizeof(double) * C)));
    t.sig = reinterpret_cast<double*>(dev(A.take(sizeof(double))));
    P.mats.push_back(t);
    for (int r = 0; r < tiles; ++r) {
      P.power[0].push_back(PowerItem{i, r, 0, 0});
      P.power[1].push_back(PowerItem{i, r, 1, 1});
      for (int c2 = 0; c2 < tiles; ++c2) {
        P.partial_items.push_back(TileItem{i, r, c2, 0});
        P.writeout_items.push_back(TileItem{i, r, c2, 0});
      }
    }
    ExpItem e{};
    e.in = m.in;
    e.ld_in = m.ld_in;
    e.a = a;
    e.out = acc;
    e.p0 = ahat;
    e.inv = inv;
    e.c = C;
    e.k = 1;
    e.size = 1;
    e.scale = 1.f;
    P.items.push_back(e);
    P.max_elems = std::max(P.max_elems, cc);
    for (int k = 2; k <= p; ++k) {
      GemmItem g{};
      g.A = k == 2 ? ahat : pp[(k - 1) & 1];
      g.B = ahat;              // A^T = -A: C = P_{k-1} Ahat = -(P_{k-1} Ahat^T)
      g.lda = g.ldb = C;
      g.K = C;
      g.M = g.N = C;
      g.C = pp[k & 1];
      g.ldc = C;
      g.dst2 = acc;
      g.ld2 = C;
      g.beta = -1.f / k;
      g.epi = EPI_SERIES;
      gemm_tiles(g, P.steps[k - 2]);
    }
  }
  P.total_bytes = align_up(A.off);
}

int validate_conv_exp(const orth_conv_exp_desc* d, int32_t n, int32_t dtype) {
  if (n < 0) return fail(ORTH_EINVAL, "n must be >= 0");
  if (n > 0 && !d) return fail(ORTH_EINVAL, "descs is NULL");
  if (dtype != ORTH_F32 && dtype != ORTH_BF16) return fail(ORTH_EINVAL, "unknown dtype");
  for (int i = 0; i < n; ++i) {
    if (!d[i].kernel || !d[i].out) return fail(ORTH_EINVAL, "NULL data pointer");
    if (d[i].channels < 1 || d[i].channels > 8192) return fail(ORTH_EINVAL, "channels must lie in [1, 8192]");
    if (d[i].k < 1 || d[i].k > 15 || d[i].k % 2 == 0) return fail(ORTH_EUNSUPPORTED, "kernel size must be odd, <= 15");
    if (d[i].terms < 1 || d[i].terms > 32) return fail(ORTH_EINVAL, "terms must lie in [1, 32]");
    if (!std::isfinite(d[i].scale)) return fail(ORTH_EINVAL, "scale must be finite");
    if (d[i].kernel == d[i].out) return fail(ORTH_EINVAL, "kernel and out must differ");
  }
  return ORTH_OK;
}

void build_conv_exp_plan(const orth_conv_exp_desc* d, int32_t n, int32_t dtype, ExpPlan& P, unsigned char* ws) {
  int max_p = 1;
  for (int i = 0; i < n; ++i) max_p = std::max(max_p, d[i].terms);
  P.steps.assign(max_p - 1, {});
  // two passes: count tables, then lay out tables followed by buffers
  for (int pass = 0; pass < 2; ++pass) {
    Arena A;
    if (pass == 1) {
      P.off_items = A.take(sizeof(ExpItem) * P.items.size());
      P.off_pairs = A.take(sizeof(GemmPair) * P.pairs.size());
      P.off_scatter = A.take(sizeof(TapItem) * P.scatter.size());
      P.off_steps.resize(P.steps.size());
      for (size_t k = 0; k < P.steps.size(); ++k) P.off_steps[k] = A.take(GemmList::bound(P.steps[k].size()));
      P.table_bytes = align_up(A.off);
      P.items.clear();
      P.pairs.clear();
      P.scatter.clear();
      for (auto& s : P.steps) s.clear();
    }
    // (pass 0 lays out from the stand-in base: its addresses are discarded)
    auto dev = [&](size_t off) -> unsigned char* { return (pass == 1 ? ws : plan_base(nullptr)) + off; };
    auto fbuf = [&](int64_t elems) { return reinterpret_cast<float*>(dev(A.take((size_t)elems * 4))); };
    for (int li = 0; li < n; ++li) {
      const orth_conv_exp_desc& L = d[li];
      const int c = L.channels, k = L.k, p = L.terms, S = p * (k - 1) + 1;
      const int64_t cc = (int64_t)c * c;
      float* lt = fbuf((int64_t)k * k * cc);
      float* acc = fbuf((int64_t)S * S * cc);
      float* q[2] = {p > 1 ? fbuf((int64_t)S * S * cc) : nullptr, p > 2 ? fbuf((int64_t)S * S * cc) : nullptr};
      ExpItem e{};
      e.in = L.kernel;
      e.a = lt;
      e.out = acc;
      e.c = c;
      e.k = k;
      e.size = S;
      e.scale = L.scale;
      P.items.push_back(e);
      P.max_elems = std::max(P.max_elems, (int64_t)k * k * cc);
      P.max_init = std::max(P.max_init, (int64_t)S * S * cc);
      for (int j = 2; j <= p; ++j) {
        const int sp = (j - 1) * (k - 1) + 1, sj = j * (k - 1) + 1, off = (S - sj) / 2;
        const float* prev = j == 2 ? lt : q[(j - 1) & 1];
        float* cur = q[j & 1];
        for (int y = 0; y < sj; ++y)
          for (int x = 0; x < sj; ++x) {
            const int base = (int)P.pairs.size();
            for (int r = 0; r < k; ++r)
              for (int t = 0; t < k; ++t) {
                const int py = y - r, px = x - t;
                if (py < 0 || py >= sp || px < 0 || px >= sp) continue;
                GemmPair gp{};
                gp.A = prev + (int64_t)(py * sp + px) * cc;
                gp.B = lt + (int64_t)((k - 1 - r) * k + (k - 1 - t)) * cc;   // L_{r,t}^T = -L_{k-1-r,k-1-t}
                gp.lda = gp.ldb = c;
                gp.K = c;
                P.pairs.push_back(gp);
              }
            GemmItem g{};
            g.pair_base = base;
            g.pair_count = (int)P.pairs.size() - base;
            g.M = g.N = c;
            g.C = cur + (int64_t)(y * sj + x) * cc;
            g.ldc = c;
            g.dst2 = acc + (int64_t)((y + off) * S + x + off) * cc;
            g.ld2 = c;
            g.beta = -1.f / j;
            g.epi = EPI_SERIES;
            gemm_tiles(g, P.steps[j - 2]);
          }
      }
      P.scatter.push_back(TapItem{acc, nullptr, L.out, nullptr, c, c, S, S, 0, 0});
      P.max_scatter = std::max(P.max_scatter, (int64_t)S * S * cc);
    }
    P.total_bytes = align_up(A.off);
  }
  (void)dtype;
}
}  // namespace

// ------------------------------------------------ Björck VJP planning ---
// The vector-Jacobian product recomputes the forward iterates, saving every
// X_t and E_t = I - X_t^T X_t (step after step in the workspace), then runs
// the gradient recurrence from t = T-1 down to 0 and finally the derivative
// of the pre-scaling.  Small matrices (N <= 64, M <= 128) run all of it in
// one workgroup each (fp32 MFMA, as in the forward); the others with fp32
// products use the fp32 tile GEMM, those with bf16 products the bf16 tile
// kernel in its saved-iterate and gradient modes.
namespace {
enum VBucket { V_F32 = 0, V_BF16_128 = 1, V_BF16_256 = 2, V_SMALL = 3 };

struct VjpPlan {
  std::vector<int> bucket;
  std::vector<TiledMat> mats;
  std::vector<TileItem> partial_items, scale_items;
  GemmList f_gram, f_upd, b_s[2], b_upd[2];
  std::vector<TileItem> t_gram[2], t_upd[2], t_s[2][2], t_yu[2][2];  // [class][parity]
  std::vector<SmallVjpMat> small[2];  // N <= 32, N <= 64 (fused kernel)
  int small_max_mp[2] = {0, 0};
  size_t off_small[2] = {0, 0};
  // spectral pre-scaling: power-step items, the backward's table of the
  // same matrices with its own vectors, and the copy of the cached vectors
  // a saving forward keeps for its saved product
  std::vector<PowerItem> power[2];
  std::vector<TiledMat> bw;
  size_t off_power[2] = {0, 0}, off_bw = 0, off_u0 = 0;
  size_t u_floats = 0;
  size_t off_mats = 0, off_partial_items = 0, off_scale_items = 0;
  size_t off_f_gram = 0, off_f_upd = 0, off_b_s[2] = {}, off_b_upd[2] = {};
  size_t off_t_gram[2] = {}, off_t_upd[2] = {}, off_t_s[2][2] = {}, off_t_yu[2][2] = {};
  size_t off_partials = 0, off_inv = 0, off_dot = 0, off_status = 0;
  size_t table_bytes = 0, total_bytes = 0;
};

void log_vjp_plan(const char* entry, const VjpPlan& P, int n) {
  if (log_level() < 1) return;
  log_line("%s: %d matrices (fused small: %zu + %zu), bf16 tiles per step: 128 %zu/%zu/%zu/%zu, 256 %zu/%zu/%zu/%zu "
           "(Gram/update/S/gradient update), fp32 64-tiles %zu/%zu/%zu/%zu; workspace %zu bytes (tables %zu)",
           entry, n, P.small[0].size(), P.small[1].size(), P.t_gram[0].size(), P.t_upd[0].size(), P.t_s[0][0].size(),
           P.t_yu[0][0].size(), P.t_gram[1].size(), P.t_upd[1].size(), P.t_s[1][0].size(), P.t_yu[1][0].size(),
           P.f_gram.size(), P.f_upd.size(), P.b_s[0].size(), P.b_upd[0].size(), P.total_bytes, P.table_bytes);
}

void seal_plan(VjpPlan& P) {
  seal(P.f_gram);
  seal(P.f_upd);
  for (int par = 0; par < 2; ++par) {
    seal(P.b_s[par]);
    seal(P.b_upd[par]);
  }
}

constexpr int kVjpMaxPowerIters = 16;

int validate_vjp(const orth_vjp_mat* mats, int32_t n, const orth_bjorck_opts* o) {
  if (n < 0) return fail(ORTH_EINVAL, "n must be >= 0");
  if (n > 0 && !mats) return fail(ORTH_EINVAL, "mats is NULL");
  if (!o) return fail(ORTH_EINVAL, "opts is NULL");
  if (o->iters < 0) return fail(ORTH_EINVAL, "iters must be >= 0");
  if (o->iters > 4096) return fail(ORTH_EINVAL, "iters must be <= 4096");
  if (!(o->beta > 0.f && o->beta <= 0.5f)) return fail(ORTH_EINVAL, "beta must lie in (0, 0.5]");
  if (o->prescale != ORTH_PRESCALE_NONE && o->prescale != ORTH_PRESCALE_FROBENIUS &&
      o->prescale != ORTH_PRESCALE_SPECTRAL)
    return fail(ORTH_EINVAL, "unknown prescale mode");
  if (o->prescale == ORTH_PRESCALE_SPECTRAL) {
    if (o->power_iters < 1 || o->power_iters > 1024) return fail(ORTH_EINVAL, "power_iters must lie in [1, 1024]");
    if (o->power_iters > kVjpMaxPowerIters)
      return fail(ORTH_EUNSUPPORTED, "the vector-Jacobian product through spectral pre-scaling takes at most 16 "
                                     "power steps");
    if (!o->u && !o->saved) return fail(ORTH_EINVAL, "spectral pre-scaling needs the cached vectors u");
  }
  if ((o->in_dtype != ORTH_F32 && o->in_dtype != ORTH_BF16) || (o->out_dtype != ORTH_F32 && o->out_dtype != ORTH_BF16))
    return fail(ORTH_EINVAL, "unknown dtype");
  if (o->compute != ORTH_COMPUTE_F32 && o->compute != ORTH_COMPUTE_BF16) return fail(ORTH_EINVAL, "unknown compute mode");
  if (o->tile != 0 && o->tile != 128 && o->tile != 256) return fail(ORTH_EINVAL, "tile must be 0, 128 or 256");
  if (o->saved != 0 && o->saved != 1) return fail(ORTH_EINVAL, "saved must be 0 or 1");
  for (int i = 0; i < n; ++i) {
    const orth_vjp_mat& m = mats[i];
    char buf[160];
    if (!m.w || !m.grad_out || !m.grad_in) {
      snprintf(buf, sizeof buf, "matrix %d: NULL data pointer", i);
      return fail(ORTH_EINVAL, buf);
    }
    if (m.rows < 1 || m.cols < 1 || m.rows > (1 << 20) || m.cols > (1 << 20)) {
      snprintf(buf, sizeof buf, "matrix %d: rows and cols must be in [1, 2^20]", i);
      return fail(ORTH_EINVAL, buf);
    }
    if (m.ld_w < m.cols || m.ld_grad_out < m.cols || m.ld_grad_in < m.cols) {
      snprintf(buf, sizeof buf, "matrix %d: leading dimension smaller than cols", i);
      return fail(ORTH_EINVAL, buf);
    }
    if (m.grad_in == m.grad_out && (o->in_dtype != o->out_dtype || m.ld_grad_in != m.ld_grad_out)) {
      snprintf(buf, sizeof buf, "matrix %d: grad_in aliasing grad_out needs equal dtypes and leading dims", i);
      return fail(ORTH_EINVAL, buf);
    }
    if (m.grad_in == m.w && m.ld_grad_in != m.ld_w) {
      snprintf(buf, sizeof buf, "matrix %d: grad_in aliasing w needs equal leading dims", i);
      return fail(ORTH_EINVAL, buf);
    }
  }
  return ORTH_OK;
}

void build_vjp_plan(const orth_vjp_mat* mats, int32_t n, const orth_bjorck_opts* o, VjpPlan& P,
                    unsigned char* ws) {
  const bool bf16 = o->compute == ORTH_COMPUTE_BF16;
  const int T = o->iters;
  const int slots = T + 1;   // X_0 .. X_T (a saving forward writes X_T too)
  const bool spectral = o->prescale == ORTH_PRESCALE_SPECTRAL;
  const int pq = spectral ? o->power_iters : 0;
  P.bucket.resize(n);
  P.mats.resize(n);
  int64_t n_part = 0, n_scale = 0, n_fg = 0, n_fu = 0, n_pw[2] = {0, 0};
  std::vector<TileItem> tg[2], tu[2];
  std::vector<int> bf16_members[2];
  std::vector<std::pair<int, int>> dims(n);
  for (int i = 0; i < n; ++i)
    dims[i] = {std::max(mats[i].rows, mats[i].cols), std::min(mats[i].rows, mats[i].cols)};
  const bool big_tiles = use_big_tiles(dims, o->tile);
  for (int i = 0; i < n; ++i) {
    const orth_vjp_mat& m = mats[i];
    TiledMat& t = P.mats[i];
    t = TiledMat{};
    t.in = m.w;
    t.out = m.grad_in;
    t.gout = m.grad_out;
    t.ld_in = m.ld_w;
    t.ld_out = m.ld_grad_in;
    t.ld_gout = m.ld_grad_out;
    t.rows = m.rows;
    t.cols = m.cols;
    t.transposed = m.rows < m.cols;
    t.M = std::max(m.rows, m.cols);
    t.N = std::min(m.rows, m.cols);
    t.status_index = i;
    int b = V_F32, pad = 64;
    if (t.N <= 64 && t.M <= 128) {
      // the whole product in one workgroup (both compute modes, as in the
      // forward): no tables, only the saved iterates
      P.bucket[i] = V_SMALL;
      t.fused = 1;
      const int k = t.N <= 32 ? 0 : 1, np = k ? 64 : 32;
      SmallVjpMat q{};
      q.w = m.w;
      q.gout = m.grad_out;
      q.gin = m.grad_in;
      q.ld_w = m.ld_w;
      q.ld_gout = m.ld_grad_out;
      q.ld_gin = m.ld_grad_in;
      q.rows = m.rows;
      q.cols = m.cols;
      q.M = t.M;
      q.N = t.N;
      q.Mp = (int32_t)round_up(t.M, 32);
      q.transposed = t.transposed;
      q.status_index = i;
      q.np = np;
      P.small[k].push_back(q);
      P.small_max_mp[k] = std::max(P.small_max_mp[k], q.Mp);
      continue;
    }
    if (bf16) {
      const bool big = t.N >= 1024 && big_tiles;
      b = big ? V_BF16_256 : V_BF16_128;
      pad = big ? 256 : 128;
    }
    P.bucket[i] = b;
    t.Mp = (int32_t)round_up(t.M, pad);
    t.Np = (int32_t)round_up(t.N, pad);
    const int pr = (m.rows + 63) / 64, pc = (m.cols + 63) / 64;
    t.partial_base = (int32_t)n_part;
    t.n_partials = pr * pc;
    n_part += pr * pc;
    n_scale += (int64_t)(t.Mp / 64) * (t.Np / 64);
    if (b == V_F32) {
      const int64_t tn = t.Np / 64, tm = t.Mp / 64;
      n_fg += tn * (tn + 1) / 2;
      n_fu += tm * tn;
    } else {
      bf16_members[b == V_BF16_256 ? 1 : 0].push_back(i);
    }
    if (spectral) {
      n_pw[0] += (t.M + 63) / 64;
      n_pw[1] += (t.N + 63) / 64;
    }
  }
  // bf16 tile lists, longest tiles first (Gram and S' tiles run over Mp,
  // update tiles over Np)
  for (int cls = 0; cls < 2; ++cls) {
    const int tsz = cls ? 256 : 128;
    std::vector<int> gm = bf16_members[cls], um = bf16_members[cls];
    std::stable_sort(gm.begin(), gm.end(), [&](int a, int c) { return P.mats[a].Mp > P.mats[c].Mp; });
    std::stable_sort(um.begin(), um.end(), [&](int a, int c) { return P.mats[a].Np > P.mats[c].Np; });
    std::vector<std::pair<int, int>> gram_mats;
    for (int i : gm) gram_mats.push_back({i, P.mats[i].Np / tsz});
    tg[cls] = bf16_gram_tiles(gram_mats);
    for (int i : um) bf16_update_tiles(i, P.mats[i].Mp / tsz, P.mats[i].Np / tsz, tu[cls]);
  }
  for (int cls = 0; cls < 2; ++cls) {
    P.t_gram[cls] = tg[cls];
    P.t_upd[cls] = tu[cls];
    for (auto& it : P.t_upd[cls]) it.flags = TILE_UPDATE;
    for (int par = 0; par < 2; ++par) {
      P.t_s[cls][par] = tg[cls];
      for (auto& it : P.t_s[cls][par]) it.flags = TILE_VJP | (par ? TILE_PARITY : 0);
      P.t_yu[cls][par] = tu[cls];
      for (auto& it : P.t_yu[cls][par]) it.flags = TILE_VJP | TILE_UPDATE | (par ? TILE_PARITY : 0);
    }
  }

  Arena A;
  P.off_mats = A.take(sizeof(TiledMat) * n);
  for (int k = 0; k < 2; ++k) P.off_small[k] = A.take(sizeof(SmallVjpMat) * P.small[k].size());
  P.off_partial_items = A.take(sizeof(TileItem) * n_part);
  P.off_scale_items = A.take(sizeof(TileItem) * n_scale);
  P.off_f_gram = A.take(GemmList::bound(n_fg));
  P.off_f_upd = A.take(GemmList::bound(n_fu));
  for (int par = 0; par < 2; ++par) {
    P.off_b_s[par] = A.take(GemmList::bound(n_fg));
    P.off_b_upd[par] = A.take(GemmList::bound(n_fu));
  }
  for (int cls = 0; cls < 2; ++cls) {
    P.off_t_gram[cls] = A.take(sizeof(TileItem) * P.t_gram[cls].size());
    P.off_t_upd[cls] = A.take(sizeof(TileItem) * P.t_upd[cls].size());
    for (int par = 0; par < 2; ++par) {
      P.off_t_s[cls][par] = A.take(sizeof(TileItem) * P.t_s[cls][par].size());
      P.off_t_yu[cls][par] = A.take(sizeof(TileItem) * P.t_yu[cls][par].size());
    }
  }
  for (int h = 0; h < 2; ++h) P.off_power[h] = A.take(sizeof(PowerItem) * n_pw[h]);
  P.off_bw = A.take(spectral ? sizeof(TiledMat) * n : 0);
  P.table_bytes = align_up(A.off);
  P.off_partials = A.take(sizeof(double) * n_part);
  P.off_inv = A.take(sizeof(float) * n);
  P.off_dot = A.take(sizeof(double) * n);
  P.off_status = A.take(sizeof(int32_t) * n);
  if (spectral)
    for (int i = 0; i < n; ++i) P.u_floats += std::min(mats[i].rows, mats[i].cols);
  P.off_u0 = A.take(sizeof(float) * P.u_floats);

  auto dev = [&](size_t off) -> unsigned char* { return ws ? ws + off : nullptr; };
  // saved X_t and E_t of the fused small matrices, pitch np
  // offsets of every matrix's cached vector in the packed array
  std::vector<int64_t> u_off(n + 1, 0);
  for (int i = 0; i < n; ++i) u_off[i + 1] = u_off[i] + (spectral ? std::min(mats[i].rows, mats[i].cols) : 0);
  const float* u_src = o->saved ? reinterpret_cast<const float*>(dev(P.off_u0)) : o->u;
  for (int k = 0; k < 2; ++k)
    for (SmallVjpMat& q : P.small[k]) {
      const int np = q.np;
      q.save = reinterpret_cast<float*>(dev(A.take((size_t)T * ((size_t)q.Mp * np + (size_t)np * np) * 4)));
      if (spectral) {
        // the start vector (the caller's u, or the saving forward's copy of
        // it), the power steps' vectors and the 2q rank-1 pairs
        q.u = u_src ? u_src + u_off[q.status_index] : nullptr;
        const size_t nd = (size_t)(pq + 1) * q.N + (size_t)pq * (q.M + q.N) + (size_t)2 * pq * (q.M + q.N);
        q.pst = reinterpret_cast<double*>(dev(A.take(sizeof(double) * nd)));
      }
    }
  std::vector<std::array<double*, 3>> bw_vec(n, {nullptr, nullptr, nullptr});
  for (int i = 0; i < n; ++i) {
    TiledMat& t = P.mats[i];
    if (t.fused) continue;
    const int64_t xe = (int64_t)t.Mp * t.Np, ee = (int64_t)t.Np * t.Np;
    t.inv_norm = reinterpret_cast<float*>(dev(P.off_inv)) + i;
    t.dot = reinterpret_cast<double*>(dev(P.off_dot)) + i;
    if (spectral) {
      auto dbl = [&](size_t cnt) { return reinterpret_cast<double*>(dev(A.take(sizeof(double) * cnt))); };
      t.u = o->u ? const_cast<float*>(o->u) + u_off[i] : nullptr;
      t.pv = dbl(t.N);
      t.px = dbl(t.M);
      t.py = dbl(t.N);
      t.sig = dbl(1);
      t.pq = pq;
      t.pst = dbl((size_t)(pq + 1) * t.N + (size_t)pq * (t.M + t.N));
      t.sb = dbl(SB_SLOTS);
      t.pair = dbl((size_t)2 * pq * (t.M + t.N));
      bw_vec[i] = {dbl(t.N), dbl(t.M), dbl(t.N)};
      // X v is a row product of W for a tall input and a column product for
      // a wide one; X^T x the other way round
      for (int b = 0; b < (t.M + 63) / 64; ++b) P.power[0].push_back(PowerItem{i, b, t.transposed, 0});
      for (int b = 0; b < (t.N + 63) / 64; ++b) P.power[1].push_back(PowerItem{i, b, !t.transposed, 1});
    }
    for (int a = 0; a < (t.rows + 63) / 64; ++a)
      for (int b = 0; b < (t.cols + 63) / 64; ++b) P.partial_items.push_back(TileItem{i, a, b, 0});
    for (int a = 0; a < t.Mp / 64; ++a)
      for (int b = 0; b < t.Np / 64; ++b) P.scale_items.push_back(TileItem{i, a, b, 0});
    if (P.bucket[i] != V_F32) {
      t.master[0] = reinterpret_cast<float*>(dev(A.take(xe * 4)));
      unsigned char* xs = dev(A.take((size_t)slots * xe * 2));
      t.xc[0] = xs;
      t.xc[1] = xs ? xs + xe * 2 : nullptr;
      t.xstep = xe;
      t.e = dev(A.take((size_t)T * ee * 2));
      t.estep = ee;
      t.gy[0] = reinterpret_cast<float*>(dev(A.take(xe * 4)));
      t.yc[0] = dev(A.take(xe * 2));
      t.yc[1] = dev(A.take(xe * 2));
      t.s = dev(A.take(ee * 2));
      t.gy_final = 0;
      continue;
    }
    // X_t and its transpose per step, E_t per step, the gradient iterate
    // and its transpose (ping-pong): every product reads row-major operands
    float* xs = reinterpret_cast<float*>(dev(A.take((size_t)slots * xe * 4)));
    float* xts = reinterpret_cast<float*>(dev(A.take((size_t)slots * xe * 4)));
    float* es = reinterpret_cast<float*>(dev(A.take((size_t)T * ee * 4)));
    float* gy0 = reinterpret_cast<float*>(dev(A.take(xe * 4)));
    float* gy1 = reinterpret_cast<float*>(dev(A.take(xe * 4)));
    float* gyt0 = reinterpret_cast<float*>(dev(A.take(xe * 4)));
    float* gyt1 = reinterpret_cast<float*>(dev(A.take(xe * 4)));
    float* sb = reinterpret_cast<float*>(dev(A.take(ee * 4)));
    t.master[0] = xs;
    t.xt = xts;
    t.e = es;
    t.gy[0] = gy0;
    t.gy[1] = gy1;
    t.gyt[0] = gyt0;
    t.gyt[1] = gyt1;
    t.s = sb;
    t.gy_final = T & 1;
    const int tn = t.Np / 64, tm = t.Mp / 64;
    for (int a = 0; a < tn; ++a)
      for (int b = a; b < tn; ++b) {
        GemmItem g{};
        g.A = xts;
        g.B = xts;
        g.lda = g.ldb = t.Mp;
        g.a_step = g.b_step = xe;
        g.K = t.Mp;
        g.M = g.N = t.Np;
        g.C = es;
        g.ldc = t.Np;
        g.c_step = ee;
        g.ti = a;
        g.tj = b;
        g.a_dtype = g.b_dtype = ORTH_F32;
        g.epi = EPI_GRAM_E;
        g.mirror = a != b;
        P.f_gram.push_back(g);
        for (int par = 0; par < 2; ++par) {
          GemmItem h{};
          h.A = xts;
          h.lda = t.Mp;
          h.a_step = xe;
          h.B = par ? gyt1 : gyt0;
          h.ldb = t.Mp;
          h.K = t.Mp;
          h.A2 = par ? gyt1 : gyt0;
          h.lda2 = t.Mp;
          h.B2 = xts;
          h.ldb2 = t.Mp;
          h.b2_step = xe;
          h.K2 = t.Mp;
          h.M = h.N = t.Np;
          h.C = sb;
          h.ldc = t.Np;
          h.ti = a;
          h.tj = b;
          h.a_dtype = h.b_dtype = ORTH_F32;
          h.epi = EPI_NEG;
          h.mirror = a != b;
          P.b_s[par].push_back(h);
        }
      }
    for (int a = 0; a < tm; ++a)
      for (int b = 0; b < tn; ++b) {
        GemmItem g{};
        g.A = xs;
        g.lda = t.Np;
        g.a_step = xe;
        g.B = es;
        g.ldb = t.Np;
        g.b_step = ee;
        g.K = t.Np;
        g.M = t.Mp;
        g.N = t.Np;
        g.src = xs;
        g.ld_src = t.Np;
        g.src_step = xe;
        g.C = xs + xe;
        g.ldc = t.Np;
        g.c_step = xe;
        g.dst2 = xts + xe;   // X_{t+1}^T
        g.ld2 = t.Mp;
        g.d2_step = xe;
        g.ti = a;
        g.tj = b;
        g.a_dtype = g.b_dtype = ORTH_F32;
        g.epi = EPI_UPDATE;
        g.beta = o->beta;
        P.f_upd.push_back(g);
        for (int par = 0; par < 2; ++par) {
          float* y = par ? gy1 : gy0;
          float* yn = par ? gy0 : gy1;
          GemmItem h{};
          h.A = y;
          h.lda = t.Np;
          h.B = es;
          h.ldb = t.Np;
          h.b_step = ee;
          h.K = t.Np;
          h.A2 = xs;
          h.lda2 = t.Np;
          h.a2_step = xe;
          h.B2 = sb;
          h.ldb2 = t.Np;
          h.K2 = t.Np;
          h.M = t.Mp;
          h.N = t.Np;
          h.src = y;
          h.ld_src = t.Np;
          h.C = yn;
          h.ldc = t.Np;
          h.dst2 = par ? gyt0 : gyt1;   // the new gradient's transpose
          h.ld2 = t.Mp;
          h.ti = a;
          h.tj = b;
          h.a_dtype = h.b_dtype = ORTH_F32;
          h.epi = EPI_UPDATE;
          h.beta = o->beta;
          P.b_upd[par].push_back(h);
        }
      }
  }
  P.total_bytes = align_up(A.off);
  if (spectral) {
    P.bw = P.mats;
    for (int i = 0; i < n; ++i) {
      P.bw[i].pv = bw_vec[i][0];
      P.bw[i].px = bw_vec[i][1];
      P.bw[i].py = bw_vec[i][2];
    }
  }
  longest_first(P.f_gram);
  longest_first(P.f_upd);
  for (int par = 0; par < 2; ++par) {
    longest_first(P.b_s[par]);
    longest_first(P.b_upd[par]);
  }
}
}  // namespace

// The orthogonalization of one batch, enqueued on `s` into the workspace
// `workspace` (at least `workspace_bytes`, checked here).  `side_streams`
// lets the small-matrix kernels run on the calling thread's side streams;
// `upload` copies the descriptor tables (nullptr: the pinned staging pool).
int ortho_enqueue(const orth_mat* mats, int32_t n, const orth_bjorck_opts* opts, void* workspace,
                  size_t workspace_bytes, int32_t* status_dev, hipStream_t s, bool side_streams,
                  TableUploader upload, const char* entry) {
  int rc = validate_ortho(mats, n, opts);
  if (rc) return rc;
  if (n == 0) return ORTH_OK;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  static PlanCache<OrthoPlan> cache;
  PlanKey key;
  key.add(n);
  key.add_bytes(mats, sizeof(orth_mat) * n);
  key.add_opts(opts);
  key.add(ws);
  const auto Pp = cache.get(key.k, [&](OrthoPlan& P) { build_ortho_plan(mats, n, opts, P, plan_base(ws), true); });
  const OrthoPlan& P = *Pp;
  rc = check_workspace(workspace, workspace_bytes, P.total_bytes);
  if (rc) return rc;
  log_ortho_plan(entry, P, opts);
  int32_t* status = status_dev ? status_dev : reinterpret_cast<int32_t*>(ws + P.off_status);

  TableImage img;
  put(img, P.off_small[0], P.small[0]);
  put(img, P.off_small[1], P.small[1]);
  put(img, P.off_tiled, P.tiled);
  put(img, P.off_partial_items, P.partial_items);
  put(img, P.off_scale_items, P.scale_items);
  put(img, P.off_writeout_items, P.writeout_items);
  for (int cls = 0; cls < 2; ++cls)
    for (int t = 0; t < N_TABS; ++t) put(img, P.off_tabs[cls][t], P.tabs[cls][t]);
  put(img, P.off_f32_gram, P.f32_gram);
  put(img, P.off_f32_update[0], P.f32_update[0]);
  put(img, P.off_f32_update[1], P.f32_update[1]);
  put(img, P.off_power[0], P.power[0]);
  put(img, P.off_power[1], P.power[1]);
  rc = upload ? upload(img.data.data(), img.spans.data(), img.spans.size(), ws, s) : upload_tables(img, ws, s);
  if (rc) return rc;

  auto T = [&](size_t off) { return reinterpret_cast<const TileItem*>(ws + off); };
  const TiledMat* tm = reinterpret_cast<const TiledMat*>(ws + P.off_tiled);
  const int nt = (int)P.tiled.size();
  const bool bf16 = opts->compute == ORTH_COMPUTE_BF16;
  const int iters = opts->iters;
  // the small-matrix kernels (one size class per side stream) run beside
  // the tiled path, which leaves most compute units idle between its
  // launches on small batches
  Fork fk(s);
  if (side_streams && nt > 0 && (!P.small[0].empty() || !P.small[1].empty())) ORTH_HIP(fk.fork());
  for (int b = 0; b < 2; ++b)
    ORTH_HIP(launch_bjorck_small(reinterpret_cast<const SmallMat*>(ws + P.off_small[b]), (int)P.small[b].size(),
                                 b ? 64 : 32, P.max_mp[b], iters, opts->beta, opts->prescale,
                                 opts->prescale == ORTH_PRESCALE_SPECTRAL ? opts->power_iters : 0, opts->in_dtype,
                                 opts->out_dtype, status, fk.side(b)));
  if (nt > 0) {
    double* partials = reinterpret_cast<double*>(ws + P.off_partials);
    ORTH_HIP(launch_prescale_partial(tm, T(P.off_partial_items), (int)P.partial_items.size(), opts->in_dtype,
                                     partials, s));
    if (opts->prescale == ORTH_PRESCALE_SPECTRAL) {
      ORTH_HIP(launch_power_init(tm, nt, s));
      for (int q = 0; q < opts->power_iters; ++q) {
        for (int h = 0; h < 2; ++h)
          ORTH_HIP(launch_power_dot(tm, reinterpret_cast<const PowerItem*>(ws + P.off_power[h]),
                                    (int)P.power[h].size(), opts->in_dtype, s));
        ORTH_HIP(launch_power_normalize(tm, nt, s));
      }
    }
    ORTH_HIP(launch_prescale_finish(tm, nt, partials, opts->prescale, status, s));
    ORTH_HIP(launch_prescale_scale(tm, T(P.off_scale_items), (int)P.scale_items.size(), opts->in_dtype,
                                   opts->compute, s));
    if (bf16) {
      // per step: all Gram tiles, then all update tiles (large class first)
      for (int t = 0; t < iters; ++t)
        for (int tab : {TAB_GRAM + (t & 1), TAB_UPDATE + (t & 1)})
          for (int cls = 1; cls >= 0; --cls)
            ORTH_HIP(launch_bf16_tiles(cls, tm, T(P.off_tabs[cls][tab]), (int)P.tabs[cls][tab].size(), opts->beta,
                                       s));
    } else {
      for (int t = 0; t < iters; ++t) {
        ORTH_HIP(launch_list(ws, P.off_f32_gram, P.f32_gram,
                                 "bjorck_gram_f32", s));
        ORTH_HIP(launch_list(ws, P.off_f32_update[t & 1], P.f32_update[t & 1], "bjorck_update_f32", s));
      }
    }
    ORTH_HIP(launch_writeout(tm, T(P.off_writeout_items), (int)P.writeout_items.size(), bf16 ? 0 : (iters & 1),
                             opts->out_dtype, s));
  }
  ORTH_HIP(fk.join());
  return ORTH_OK;
}

}  // namespace orth

using namespace orth;

// ================================================================== C ABI =
extern "C" {

const char* orth_status_string(int status) {
  switch (status) {
    case ORTH_OK: return "ok";
    case ORTH_EINVAL: return "invalid argument";
    case ORTH_EUNSUPPORTED: return "unsupported configuration";
    case ORTH_EWORKSPACE: return "workspace missing, too small or misaligned";
    case ORTH_EHIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* orth_last_error(void) { return g_last_error.c_str(); }

int32_t orth_version(void) { return 100; }

int orth_orthogonalize_workspace_size(const orth_mat* mats, int32_t n, const orth_bjorck_opts* opts,
                                      size_t* bytes) {
  if (!bytes) return fail(ORTH_EINVAL, "bytes is NULL");
  int rc = validate_ortho(mats, n, opts);
  if (rc) return rc;
  OrthoPlan P;
  build_ortho_plan(mats, n, opts, P, plan_base(nullptr), true);
  *bytes = P.total_bytes;
  return ORTH_OK;
}

int orth_orthogonalize_batched(const orth_mat* mats, int32_t n, const orth_bjorck_opts* opts, void* workspace,
                               size_t workspace_bytes, int32_t* status_dev, void* stream) {
  return ortho_enqueue(mats, n, opts, workspace, workspace_bytes, status_dev, static_cast<hipStream_t>(stream), true,
                       nullptr, "orth_orthogonalize_batched");
}

namespace {
// Pre-scaling and the forward steps of a vector-Jacobian product plan, with
// X_t and E_t of every step left in the workspace.  `to_output` also runs
// the last update and writes X_T to the plan's output (a saving forward).
int vjp_forward(const VjpPlan& P, unsigned char* ws, const orth_bjorck_opts* opts, int n, int32_t* status,
                bool to_output, hipStream_t s) {
  auto TI = [&](size_t off) { return reinterpret_cast<const TileItem*>(ws + off); };
  const TiledMat* tm = reinterpret_cast<const TiledMat*>(ws + P.off_mats);
  const int T = opts->iters;
  const float beta = opts->beta;
  double* partials = reinterpret_cast<double*>(ws + P.off_partials);
  ORTH_HIP(launch_prescale_partial(tm, TI(P.off_partial_items), (int)P.partial_items.size(), opts->in_dtype,
                                   partials, s));
  if (opts->prescale == ORTH_PRESCALE_SPECTRAL) {
    // the power steps, every step's vectors kept for the backward
    ORTH_HIP(launch_power_init(tm, n, s));
    ORTH_HIP(launch_power_keep(tm, n, 0, s));
    for (int k = 1; k <= opts->power_iters; ++k) {
      for (int h = 0; h < 2; ++h)
        ORTH_HIP(launch_power_dot(tm, reinterpret_cast<const PowerItem*>(ws + P.off_power[h]),
                                  (int)P.power[h].size(), opts->in_dtype, s));
      ORTH_HIP(launch_power_normalize(tm, n, s));
      ORTH_HIP(launch_power_keep(tm, n, k, s));
    }
  }
  // a saving forward hands the new estimate back; the recomputation inside
  // a vector-Jacobian product leaves the cached vectors alone
  ORTH_HIP(launch_prescale_finish(tm, n, partials, opts->prescale, status, s, to_output ? 1 : 0));
  ORTH_HIP(launch_prescale_scale(tm, TI(P.off_scale_items), (int)P.scale_items.size(), opts->in_dtype,
                                 opts->compute, s));
  for (int t = 0; t < T; ++t) {
    ORTH_HIP(launch_list(ws, P.off_f_gram, P.f_gram, "vjp_fwd_gram_f32", s, t));
    for (int cls = 1; cls >= 0; --cls)
      ORTH_HIP(launch_bf16_tiles(cls, tm, TI(P.off_t_gram[cls]), (int)P.t_gram[cls].size(), beta, s, 0, t));
    if (t + 1 == T && !to_output) break;
    ORTH_HIP(launch_list(ws, P.off_f_upd, P.f_upd, "vjp_fwd_update_f32", s, t));
    for (int cls = 1; cls >= 0; --cls)
      ORTH_HIP(launch_bf16_tiles(cls, tm, TI(P.off_t_upd[cls]), (int)P.t_upd[cls].size(), beta, s, 0, t));
  }
  if (to_output)   // master[1] of every tiled matrix points at X_T (fp32)
    ORTH_HIP(launch_writeout(tm, TI(P.off_partial_items), (int)P.partial_items.size(), 1, opts->out_dtype, s));
  return ORTH_OK;
}

// The vector-Jacobian descriptors whose plan a saving forward shares: w is
// the forward's input, grad_in its output (the plan's output slot) and
// grad_out a placeholder never read by the forward part.
int save_descs(const orth_mat* mats, int32_t n, const orth_bjorck_opts* opts, std::vector<orth_vjp_mat>& vm) {
  int rc = validate_ortho(mats, n, opts);
  if (rc) return rc;
  if (opts->saved) return fail(ORTH_EINVAL, "saved must be 0 for the saving forward");
  vm.resize(n);
  for (int i = 0; i < n; ++i) {
    const orth_mat& m = mats[i];
    if (m.in == m.out) {
      char buf[160];
      snprintf(buf, sizeof buf, "matrix %d: a saving forward cannot run in place (the VJP reads the input)", i);
      return fail(ORTH_EINVAL, buf);
    }
    vm[i] = orth_vjp_mat{m.in, m.in, m.out, m.rows, m.cols, m.ld_in, m.ld_in, m.ld_out};
  }
  return validate_vjp(vm.data(), n, opts);
}
}  // namespace

int orth_orthogonalize_save_workspace_size(const orth_mat* mats, int32_t n, const orth_bjorck_opts* opts,
                                           size_t* bytes) {
  if (!bytes) return fail(ORTH_EINVAL, "bytes is NULL");
  std::vector<orth_vjp_mat> vm;
  int rc = save_descs(mats, n, opts, vm);
  if (rc) return rc;
  VjpPlan P;
  build_vjp_plan(vm.data(), n, opts, P, plan_base(nullptr));
  *bytes = P.total_bytes;
  return ORTH_OK;
}

int orth_orthogonalize_save_batched(const orth_mat* mats, int32_t n, const orth_bjorck_opts* opts, void* workspace,
                                    size_t workspace_bytes, int32_t* status_dev, void* stream) {
  std::vector<orth_vjp_mat> vm;
  int rc = save_descs(mats, n, opts, vm);
  if (rc) return rc;
  if (n == 0) return ORTH_OK;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  static PlanCache<VjpPlan> cache;
  PlanKey key;
  key.add(n);
  key.add_bytes(vm.data(), sizeof(orth_vjp_mat) * n);
  key.add_opts(opts);
  key.add(ws);
  const auto Pp = cache.get(key.k, [&](VjpPlan& P) { build_vjp_plan(vm.data(), n, opts, P, plan_base(ws)); });
  const VjpPlan& P = *Pp;
  rc = check_workspace(workspace, workspace_bytes, P.total_bytes);
  if (rc) return rc;
  log_vjp_plan("orth_orthogonalize_save_batched", P, n);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // statuses go to the workspace, where the saved product reads them, and
  // are copied to the caller's array
  int32_t* status = reinterpret_cast<int32_t*>(ws + P.off_status);
  // X_T of a tiled matrix: the fp32 iterate (bf16 products, updated in
  // place) or saved slot T (fp32 products)
  std::vector<TiledMat> fwd_mats = P.mats;
  for (int i = 0; i < n; ++i) {
    TiledMat& t = fwd_mats[i];
    if (t.fused) continue;
    t.master[1] = P.bucket[i] == V_F32 ? t.master[0] + (int64_t)opts->iters * t.Mp * t.Np : t.master[0];
  }
  // small matrices: the forward kernel, its table in the place of the
  // vector-Jacobian one
  static_assert(sizeof(SmallMat) <= sizeof(SmallVjpMat), "small tables share their workspace region");
  std::vector<SmallMat> small[2];
  for (int k = 0; k < 2; ++k)
    for (const SmallVjpMat& q : P.small[k]) {
      SmallMat sm{};
      sm.in = q.w;
      sm.out = q.gin;
      sm.ld_in = q.ld_w;
      sm.ld_out = q.ld_gin;
      sm.rows = q.rows;
      sm.cols = q.cols;
      sm.M = q.M;
      sm.N = q.N;
      sm.Mp = q.Mp;
      sm.transposed = q.transposed;
      sm.status_index = q.status_index;
      sm.u = const_cast<float*>(q.u);
      small[k].push_back(sm);
    }
  TableImage img;
  put(img, P.off_mats, fwd_mats);
  for (int k = 0; k < 2; ++k) put(img, P.off_small[k], small[k]);
  put(img, P.off_power[0], P.power[0]);
  put(img, P.off_power[1], P.power[1]);
  put(img, P.off_bw, P.bw);
  put(img, P.off_partial_items, P.partial_items);
  put(img, P.off_scale_items, P.scale_items);
  put(img, P.off_f_gram, P.f_gram);
  put(img, P.off_f_upd, P.f_upd);
  for (int cls = 0; cls < 2; ++cls) {
    put(img, P.off_t_gram[cls], P.t_gram[cls]);
    put(img, P.off_t_upd[cls], P.t_upd[cls]);
  }
  rc = upload_tables(img, ws, s);
  if (rc) return rc;
  // spectral: the cached vectors as this call found them, for the saved
  // product (this call writes the new estimates back into u)
  if (opts->prescale == ORTH_PRESCALE_SPECTRAL && P.u_floats)
    ORTH_HIP(hipMemcpyAsync(ws + P.off_u0, opts->u, sizeof(float) * P.u_floats, hipMemcpyDeviceToDevice, s));
  // small matrices on side streams beside the tiled forward
  Fork fk(s);
  if (!P.partial_items.empty() && (!small[0].empty() || !small[1].empty())) ORTH_HIP(fk.fork());
  for (int k = 0; k < 2; ++k)
    ORTH_HIP(launch_bjorck_small(reinterpret_cast<const SmallMat*>(ws + P.off_small[k]), (int)small[k].size(),
                                 k ? 64 : 32, P.small_max_mp[k], opts->iters, opts->beta, opts->prescale,
                                 opts->prescale == ORTH_PRESCALE_SPECTRAL ? opts->power_iters : 0,
                                 opts->in_dtype, opts->out_dtype, status, fk.side(k)));
  rc = vjp_forward(P, ws, opts, n, status, true, s);
  if (rc) return rc;
  ORTH_HIP(fk.join());
  if (status_dev) ORTH_HIP(hipMemcpyAsync(status_dev, status, sizeof(int32_t) * n, hipMemcpyDeviceToDevice, s));
  return ORTH_OK;
}

int orth_orthogonalize_vjp_workspace_size(const orth_vjp_mat* mats, int32_t n, const orth_bjorck_opts* opts,
                                          size_t* bytes) {
  if (!bytes) return fail(ORTH_EINVAL, "bytes is NULL");
  int rc = validate_vjp(mats, n, opts);
  if (rc) return rc;
  VjpPlan P;
  build_vjp_plan(mats, n, opts, P, plan_base(nullptr));
  *bytes = P.total_bytes;
  return ORTH_OK;
}

int orth_orthogonalize_vjp_batched(const orth_vjp_mat* mats, int32_t n, const orth_bjorck_opts* opts,
                                   void* workspace, size_t workspace_bytes, int32_t* status_dev, void* stream) {
  int rc = validate_vjp(mats, n, opts);
  if (rc) return rc;
  if (n == 0) return ORTH_OK;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  static PlanCache<VjpPlan> cache;
  PlanKey key;
  key.add(n);
  key.add_bytes(mats, sizeof(orth_vjp_mat) * n);
  key.add_opts(opts);
  key.add(ws);
  const auto Pp = cache.get(key.k, [&](VjpPlan& P) { build_vjp_plan(mats, n, opts, P, plan_base(ws)); });
  const VjpPlan& P = *Pp;
  rc = check_workspace(workspace, workspace_bytes, P.total_bytes);
  if (rc) return rc;
  log_vjp_plan("orth_orthogonalize_vjp_batched", P, n);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // with saved iterates the statuses of the saving forward are in the
  // workspace; the small-matrix kernel refreshes its own
  int32_t* status =
      status_dev && !opts->saved ? status_dev : reinterpret_cast<int32_t*>(ws + P.off_status);

  TableImage img;
  put(img, P.off_mats, P.mats);
  for (int k = 0; k < 2; ++k) put(img, P.off_small[k], P.small[k]);
  put(img, P.off_power[0], P.power[0]);
  put(img, P.off_power[1], P.power[1]);
  put(img, P.off_bw, P.bw);
  put(img, P.off_partial_items, P.partial_items);
  put(img, P.off_scale_items, P.scale_items);
  put(img, P.off_f_gram, P.f_gram);
  put(img, P.off_f_upd, P.f_upd);
  for (int par = 0; par < 2; ++par) {
    put(img, P.off_b_s[par], P.b_s[par]);
    put(img, P.off_b_upd[par], P.b_upd[par]);
  }
  for (int cls = 0; cls < 2; ++cls) {
    put(img, P.off_t_gram[cls], P.t_gram[cls]);
    put(img, P.off_t_upd[cls], P.t_upd[cls]);
    for (int par = 0; par < 2; ++par) {
      put(img, P.off_t_s[cls][par], P.t_s[cls][par]);
      put(img, P.off_t_yu[cls][par], P.t_yu[cls][par]);
    }
  }
  rc = upload_tables(img, ws, s);
  if (rc) return rc;

  auto TI = [&](size_t off) { return reinterpret_cast<const TileItem*>(ws + off); };
  const TiledMat* tm = reinterpret_cast<const TiledMat*>(ws + P.off_mats);
  const int T = opts->iters;
  const float beta = opts->beta;
  double* partials = reinterpret_cast<double*>(ws + P.off_partials);
  // small matrices: the whole product per workgroup, on side streams
  // beside the tiled matrices' steps
  Fork fk(s);
  if (!P.partial_items.empty() && (!P.small[0].empty() || !P.small[1].empty())) ORTH_HIP(fk.fork());
  for (int k = 0; k < 2; ++k)
    ORTH_HIP(launch_bjorck_small_vjp(reinterpret_cast<const SmallVjpMat*>(ws + P.off_small[k]),
                                     (int)P.small[k].size(), k ? 64 : 32, P.small_max_mp[k], T, beta,
                                     opts->prescale,
                                     opts->prescale == ORTH_PRESCALE_SPECTRAL ? opts->power_iters : 0,
                                     opts->in_dtype, opts->out_dtype, status, fk.side(k)));
  // forward recomputation, saving X_t and E_t (X_T itself is never
  // needed), unless a saving forward left them in the workspace
  if (!opts->saved) {
    rc = vjp_forward(P, ws, opts, n, status, false, s);
    if (rc) return rc;
  }
  // gradient recurrence, last step first
  ORTH_HIP(launch_vjp_load_grad(tm, TI(P.off_scale_items), (int)P.scale_items.size(), opts->out_dtype, s));
  for (int b = 0; b < T; ++b) {
    const int t = T - 1 - b, par = b & 1;
    ORTH_HIP(launch_list(ws, P.off_b_s[par], P.b_s[par], "vjp_s_f32", s, t));
    for (int cls = 1; cls >= 0; --cls)
      ORTH_HIP(launch_bf16_tiles(cls, tm, TI(P.off_t_s[cls][par]), (int)P.t_s[cls][par].size(), beta, s, 1, t));
    ORTH_HIP(launch_list(ws, P.off_b_upd[par], P.b_upd[par], "vjp_update_f32", s, t));
    for (int cls = 1; cls >= 0; --cls)
      ORTH_HIP(launch_bf16_tiles(cls, tm, TI(P.off_t_yu[cls][par]), (int)P.t_yu[cls][par].size(), beta, s, 1, t));
  }
  // derivative of the pre-scaling, in the caller's layout
  if (opts->prescale != ORTH_PRESCALE_NONE) {
    ORTH_HIP(launch_vjp_dot_partial(tm, TI(P.off_partial_items), (int)P.partial_items.size(), opts->in_dtype,
                                    partials, s));
    ORTH_HIP(launch_vjp_dot_finish(tm, n, partials, s));
  }
  if (opts->prescale == ORTH_PRESCALE_SPECTRAL)
    ORTH_HIP(launch_spec_bwd(tm, reinterpret_cast<const TiledMat*>(ws + P.off_bw), n,
                             reinterpret_cast<const PowerItem*>(ws + P.off_power[0]), (int)P.power[0].size(),
                             reinterpret_cast<const PowerItem*>(ws + P.off_power[1]), (int)P.power[1].size(),
                             opts->power_iters, opts->in_dtype, status, s));
  ORTH_HIP(launch_vjp_writeout(tm, TI(P.off_partial_items), (int)P.partial_items.size(), opts->in_dtype,
                               opts->prescale, status, s));
  ORTH_HIP(fk.join());
  if (opts->saved && status_dev)
    ORTH_HIP(hipMemcpyAsync(status_dev, status, sizeof(int32_t) * n, hipMemcpyDeviceToDevice, s));
  return ORTH_OK;
}

int orth_aoc_param_shapes(const orth_conv_geom* geom, int32_t* rko_rows, int32_t* rko_cols, int32_t* n_proj,
                          int32_t* proj_rows, int32_t* proj_cols) {
  const int rc = validate_geom(geom);
  if (rc) return rc;
  const int c = geom->cin / geom->groups, s = geom->stride;
  if (rko_rows) *rko_rows = geom->cout / geom->groups;
  if (rko_cols) *rko_cols = c * s * s;
  if (n_proj) *n_proj = 2 * (geom->k - s);
  if (proj_rows) *proj_rows = c;
  if (proj_cols) *proj_cols = c / 2;
  return ORTH_OK;
}

int orth_build_conv_kernels_workspace_size(const orth_conv_desc* descs, int32_t n, int32_t dtype, size_t* bytes) {
  if (!bytes) return fail(ORTH_EINVAL, "bytes is NULL");
  int rc = validate_conv_descs(descs, n, dtype);
  if (rc) return rc;
  ConvPlan P;
  build_conv_plan(descs, n, dtype, P, plan_base(nullptr));
  *bytes = P.total_bytes;
  return ORTH_OK;
}

int orth_build_conv_kernels_batched(const orth_conv_desc* descs, int32_t n, int32_t dtype, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  int rc = validate_conv_descs(descs, n, dtype);
  if (rc) return rc;
  if (n == 0) return ORTH_OK;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  static PlanCache<ConvPlan> cache;
  PlanKey key;
  key.add(n);
  key.add(dtype);
  key.add_bytes(descs, sizeof(orth_conv_desc) * n);
  key.add(ws);
  const auto Pp = cache.get(key.k, [&](ConvPlan& P) { build_conv_plan(descs, n, dtype, P, plan_base(ws)); });
  const ConvPlan& P = *Pp;
  rc = check_workspace(workspace, workspace_bytes, P.total_bytes);
  if (rc) return rc;
  if (log_level() >= 1) {
    size_t tiles = P.proj_items.size();
    for (const auto& g : P.phase_gemm) tiles += g.size();
    log_line("orth_build_conv_kernels_batched: %d layers, %zu groups, %zu block steps, %zu fp32 64-tiles; "
             "workspace %zu bytes (tables %zu)", n, P.groups.size(), P.phase_gemm.size(), tiles, P.total_bytes,
             P.table_bytes);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);

  TableImage img;
  put(img, P.off_groups, P.groups);
  put(img, P.off_proj_items, P.proj_items);
  for (size_t ph = 0; ph < P.phase_gemm.size(); ++ph) {
    put(img, P.off_phase_gemm[ph], P.phase_gemm[ph]);
    put(img, P.off_phase_comb[ph], P.phase_comb[ph]);
  }
  put(img, P.off_scatter, P.scatter);
  rc = upload_tables(img, ws, s);
  if (rc) return rc;
  const ComposeGroup* G = reinterpret_cast<const ComposeGroup*>(ws + P.off_groups);
  const int ng = (int)P.groups.size();
  ORTH_HIP(launch_compose_init(G, ng, dtype, P.init_max, s));
  ORTH_HIP(launch_list(ws, P.off_proj_items, P.proj_items, "compose_projector", s));
  for (size_t ph = 0; ph < P.phase_gemm.size(); ++ph) {
    ORTH_HIP(launch_list(ws, P.off_phase_gemm[ph], P.phase_gemm[ph], "compose_tap_gemm", s));
    ORTH_HIP(launch_compose_combine(G, reinterpret_cast<const CombineItem*>(ws + P.off_phase_comb[ph]),
                                    (int)P.phase_comb[ph].size(), P.phase_max_elems[ph], s));
  }
  ORTH_HIP(launch_tap_items(2, reinterpret_cast<const TapItem*>(ws + P.off_scatter), (int)P.scatter.size(), dtype,
                            P.scatter_max, s, "compose_scatter"));
  return ORTH_OK;
}

int orth_build_conv_kernels_vjp_workspace_size(const orth_conv_vjp_desc* descs, int32_t n, int32_t dtype,
                                               size_t* bytes) {
  if (!bytes) return fail(ORTH_EINVAL, "bytes is NULL");
  const int rc = validate_conv_vjp_descs(descs, n, dtype);
  if (rc) return rc;
  ConvVjpPlan P;
  build_conv_vjp_plan(descs, n, dtype, P, plan_base(nullptr));
  *bytes = P.total_bytes;
  return ORTH_OK;
}

namespace {
// mode 0: vector-Jacobian product with the forward recomputed; 1: the same
// from the tap grids and projectors a saving forward left in the workspace;
// 2: the saving forward (kernels[] receive the composed kernels)
int conv_vjp_run(const orth_conv_vjp_desc* descs, int32_t n, int32_t dtype, void* workspace,
                 size_t workspace_bytes, void* stream, int mode, const void* const* kernels) {
  if (n == 0) return ORTH_OK;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  static PlanCache<ConvVjpPlan> cache;
  PlanKey key;
  key.add(n);
  key.add(dtype);
  key.add(mode);
  key.add_bytes(descs, sizeof(orth_conv_vjp_desc) * n);
  key.add_bytes(kernels, kernels ? sizeof(void*) * n : 0);
  key.add(ws);
  const auto Pp =
      cache.get(key.k, [&](ConvVjpPlan& P) { build_conv_vjp_plan(descs, n, dtype, P, plan_base(ws), kernels); });
  const ConvVjpPlan& P = *Pp;
  int rc = check_workspace(workspace, workspace_bytes, P.total_bytes);
  if (rc) return rc;
  if (log_level() >= 1)
    log_line("composition VJP (mode %d): %d layers, %zu block steps; workspace %zu bytes (tables %zu)", mode, n,
             P.fwd_gemm.size(), P.total_bytes, P.table_bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int n_phase = (int)P.fwd_gemm.size();

  TableImage img;
  put(img, P.off_proj, P.proj_items);
  put(img, P.off_last_dp, P.last_dp);
  put(img, P.off_dv, P.dv_items);
  put(img, P.off_rko_taps, P.rko_taps);
  put(img, P.off_grad_taps, P.grad_taps);
  put(img, P.off_rko_grad, P.rko_grad);
  put(img, P.off_save_scatter, P.save_scatter);
  for (int ph = 0; ph < n_phase; ++ph) {
    put(img, P.off_fwd_gemm[ph], P.fwd_gemm[ph]);
    put(img, P.off_bwd_gemm[ph], P.bwd_gemm[ph]);
    put(img, P.off_fwd_comb[ph], P.fwd_comb[ph]);
    put(img, P.off_bwd_comb[ph], P.bwd_comb[ph]);
    put(img, P.off_save_gemm[ph], P.save_gemm[ph]);
    put(img, P.off_save_comb[ph], P.save_comb[ph]);
  }
  rc = upload_tables(img, ws, s);
  if (rc) return rc;
  auto TI = [&](size_t off) { return reinterpret_cast<const TapItem*>(ws + off); };
  if (mode != 1) {
    // forward: RKO taps, projectors, the block steps (keeping every input grid)
    ORTH_HIP(launch_tap_items(0, TI(P.off_rko_taps), (int)P.rko_taps.size(), dtype, P.rko_max, s));
    ORTH_HIP(launch_list(ws, P.off_proj, P.proj_items, "conv_vjp_projector", s));
    for (int ph = 0; ph < n_phase; ++ph) {
      ORTH_HIP(launch_list(ws, P.off_fwd_gemm[ph], P.fwd_gemm[ph], "conv_vjp_tap_gemm", s));
      if (mode == 2) ORTH_HIP(launch_list(ws, P.off_save_gemm[ph], P.save_gemm[ph], "conv_vjp_tap_gemm", s));
      ORTH_HIP(launch_tap_items(3, TI(P.off_fwd_comb[ph]), (int)P.fwd_comb[ph].size(), dtype, P.fwd_max[ph], s));
      if (mode == 2)
        ORTH_HIP(launch_tap_items(3, TI(P.off_save_comb[ph]), (int)P.save_comb[ph].size(), dtype, P.save_max[ph], s));
    }
  }
  if (mode == 2) {
    ORTH_HIP(launch_tap_items(2, TI(P.off_save_scatter), (int)P.save_scatter.size(), dtype, P.scatter_max, s));
    return ORTH_OK;
  }
  ORTH_HIP(launch_tap_items(1, TI(P.off_grad_taps), (int)P.grad_taps.size(), dtype, P.grad_max, s));
  for (int ph = n_phase - 1; ph >= 0; --ph) {
    ORTH_HIP(launch_list(ws, P.off_bwd_gemm[ph], P.bwd_gemm[ph], "conv_vjp_tap_gemm", s));
    ORTH_HIP(launch_tap_items(4, TI(P.off_bwd_comb[ph]), (int)P.bwd_comb[ph].size(), dtype, P.bwd_max[ph], s));
  }
  ORTH_HIP(launch_list(ws, P.off_last_dp, P.last_dp, "conv_vjp_tap_gemm", s));
  ORTH_HIP(launch_list(ws, P.off_dv, P.dv_items, "conv_vjp_factor_grad", s));
  ORTH_HIP(launch_tap_items(2, TI(P.off_rko_grad), (int)P.rko_grad.size(), dtype, P.rko_max, s));
  return ORTH_OK;
}

// The vector-Jacobian descriptors whose plan a saving composition shares:
// the gradient fields hold placeholders that the forward never touches.
int conv_save_descs(const orth_conv_desc* d, int32_t n, int32_t dtype, std::vector<orth_conv_vjp_desc>& vd,
                    std::vector<const void*>& kernels) {
  int rc = validate_conv_descs(d, n, dtype);
  if (rc) return rc;
  vd.resize(n);
  kernels.resize(n);
  for (int i = 0; i < n; ++i) {
    vd[i] = orth_conv_vjp_desc{};
    vd[i].geom = d[i].geom;
    vd[i].rko = d[i].rko;
    vd[i].proj = d[i].proj;
    vd[i].grad_kernel = d[i].kernel;
    vd[i].grad_rko = const_cast<void*>(d[i].rko);
    vd[i].grad_proj = const_cast<void*>(d[i].proj);
    kernels[i] = d[i].kernel;
  }
  return validate_conv_vjp_descs(vd.data(), n, dtype);
}
}  // namespace

int orth_build_conv_kernels_vjp_batched(const orth_conv_vjp_desc* descs, int32_t n, int32_t dtype, void* workspace,
                                        size_t workspace_bytes, void* stream) {
  const int rc = validate_conv_vjp_descs(descs, n, dtype);
  if (rc) return rc;
  return conv_vjp_run(descs, n, dtype, workspace, workspace_bytes, stream, 0, nullptr);
}

int orth_build_conv_kernels_vjp_saved_batched(const orth_conv_vjp_desc* descs, int32_t n, int32_t dtype,
                                              void* workspace, size_t workspace_bytes, void* stream) {
  const int rc = validate_conv_vjp_descs(descs, n, dtype);
  if (rc) return rc;
  return conv_vjp_run(descs, n, dtype, workspace, workspace_bytes, stream, 1, nullptr);
}

int orth_build_conv_kernels_save_workspace_size(const orth_conv_desc* descs, int32_t n, int32_t dtype,
                                                size_t* bytes) {
  if (!bytes) return fail(ORTH_EINVAL, "bytes is NULL");
  std::vector<orth_conv_vjp_desc> vd;
  std::vector<const void*> kernels;
  const int rc = conv_save_descs(descs, n, dtype, vd, kernels);
  if (rc) return rc;
  ConvVjpPlan P;
  build_conv_vjp_plan(vd.data(), n, dtype, P, plan_base(nullptr));
  *bytes = P.total_bytes;
  return ORTH_OK;
}

int orth_build_conv_kernels_save_batched(const orth_conv_desc* descs, int32_t n, int32_t dtype, void* workspace,
                                         size_t workspace_bytes, void* stream) {
  std::vector<orth_conv_vjp_desc> vd;
  std::vector<const void*> kernels;
  const int rc = conv_save_descs(descs, n, dtype, vd, kernels);
  if (rc) return rc;
  return conv_vjp_run(vd.data(), n, dtype, workspace, workspace_bytes, stream, 2, kernels.data());
}

int orth_conv_apply(const orth_conv_apply_args* a, void* stream) {
  if (!a) return fail(ORTH_EINVAL, "args is NULL");
  const int rc = validate_geom(&a->geom);
  if (rc) return rc;
  if (!a->kernel || !a->x || !a->y) return fail(ORTH_EINVAL, "NULL data pointer");
  if (static_cast<const void*>(a->x) == static_cast<const void*>(a->y)) return fail(ORTH_EINVAL, "x and y must differ");
  if (a->kernel_dtype != ORTH_F32 && a->kernel_dtype != ORTH_BF16) return fail(ORTH_EINVAL, "unknown dtype");
  if (a->batch < 1 || a->height < 1 || a->width < 1) return fail(ORTH_EINVAL, "batch, height and width must be >= 1");
  if (a->height % a->geom.stride || a->width % a->geom.stride)
    return fail(ORTH_EINVAL, "height and width must be divisible by the stride");
  const int64_t pix = (int64_t)a->batch * a->height * a->width;
  if (pix / 64 + 1 > INT32_MAX) return fail(ORTH_EINVAL, "batch x height x width too large");
  ORTH_HIP(launch_conv_apply(a, static_cast<hipStream_t>(stream)));
  return ORTH_OK;
}

int orth_exp_map_workspace_size(const orth_mat* mats, int32_t n, const orth_exp_opts* opts, size_t* bytes) {
  if (!bytes) return fail(ORTH_EINVAL, "bytes is NULL");
  const int rc = validate_exp(mats, n, opts);
  if (rc) return rc;
  ExpPlan P;
  build_exp_plan(mats, n, opts, P, plan_base(nullptr));
  *bytes = P.total_bytes;
  return ORTH_OK;
}

int orth_exp_map_batched(const orth_mat* mats, int32_t n, const orth_exp_opts* opts, void* workspace,
                         size_t workspace_bytes, int32_t* status_dev, void* stream) {
  int rc = validate_exp(mats, n, opts);
  if (rc) return rc;
  if (n == 0) return ORTH_OK;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  ExpPlan P;
  build_exp_plan(mats, n, opts, P, plan_base(ws));
  rc = check_workspace(workspace, workspace_bytes, P.total_bytes);
  if (rc) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t* status = status_dev ? status_dev : reinterpret_cast<int32_t*>(ws + P.off_status);
  TableImage img;
  put(img, P.off_items, P.items);
  put(img, P.off_mats, P.mats);
  put(img, P.off_partial, P.partial_items);
  put(img, P.off_writeout, P.writeout_items);
  put(img, P.off_power[0], P.power[0]);
  put(img, P.off_power[1], P.power[1]);
  for (size_t k = 0; k < P.steps.size(); ++k) put(img, P.off_steps[k], P.steps[k]);
  rc = upload_tables(img, ws, s);
  if (rc) return rc;
  const ExpItem* items = reinterpret_cast<const ExpItem*>(ws + P.off_items);
  const TiledMat* tm = reinterpret_cast<const TiledMat*>(ws + P.off_mats);
  auto TI = [&](size_t off) { return reinterpret_cast<const TileItem*>(ws + off); };
  double* partials = reinterpret_cast<double*>(ws + P.off_partials);
  ORTH_HIP(launch_exp_skew(items, n, 0, opts->in_dtype, P.max_elems, s));
  // spectral normalization of A (the fp32 A in the workspace is the input)
  ORTH_HIP(launch_prescale_partial(tm, TI(P.off_partial), (int)P.partial_items.size(), ORTH_F32, partials, s));
  ORTH_HIP(launch_power_init(tm, n, s));
  for (int q = 0; q < opts->power_iters; ++q) {
    for (int h = 0; h < 2; ++h)
      ORTH_HIP(launch_power_dot(tm, reinterpret_cast<const PowerItem*>(ws + P.off_power[h]), (int)P.power[h].size(),
                                ORTH_F32, s));
    ORTH_HIP(launch_power_normalize(tm, n, s));
  }
  ORTH_HIP(launch_prescale_finish(tm, n, partials, ORTH_PRESCALE_SPECTRAL, status, s));
  ORTH_HIP(launch_exp_init(items, n, 0, P.max_elems, s));
  for (size_t k = 0; k < P.steps.size(); ++k)
    ORTH_HIP(launch_list(ws, P.off_steps[k], P.steps[k], "exp_map_series", s));
  ORTH_HIP(launch_writeout(tm, TI(P.off_writeout), (int)P.writeout_items.size(), 0, opts->out_dtype, s));
  return ORTH_OK;
}

int orth_conv_exp_workspace_size(const orth_conv_exp_desc* descs, int32_t n, int32_t dtype, size_t* bytes) {
  if (!bytes) return fail(ORTH_EINVAL, "bytes is NULL");
  const int rc = validate_conv_exp(descs, n, dtype);
  if (rc) return rc;
  ExpPlan P;
  build_conv_exp_plan(descs, n, dtype, P, plan_base(nullptr));
  *bytes = P.total_bytes;
  return ORTH_OK;
}

int orth_conv_exp_batched(const orth_conv_exp_desc* descs, int32_t n, int32_t dtype, void* workspace,
                          size_t workspace_bytes, void* stream) {
  int rc = validate_conv_exp(descs, n, dtype);
  if (rc) return rc;
  if (n == 0) return ORTH_OK;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  ExpPlan P;
  build_conv_exp_plan(descs, n, dtype, P, plan_base(ws));
  rc = check_workspace(workspace, workspace_bytes, P.total_bytes);
  if (rc) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  TableImage img;
  put(img, P.off_items, P.items);
  put(img, P.off_pairs, P.pairs);
  put(img, P.off_scatter, P.scatter);
  for (size_t k = 0; k < P.steps.size(); ++k) put(img, P.off_steps[k], P.steps[k]);
  rc = upload_tables(img, ws, s);
  if (rc) return rc;
  const ExpItem* items = reinterpret_cast<const ExpItem*>(ws + P.off_items);
  ORTH_HIP(launch_exp_skew(items, n, 1, dtype, P.max_elems, s));
  ORTH_HIP(launch_exp_init(items, n, 1, P.max_init, s));
  const GemmPair* pairs = reinterpret_cast<const GemmPair*>(ws + P.off_pairs);
  for (size_t k = 0; k < P.steps.size(); ++k)
    ORTH_HIP(launch_list(ws, P.off_steps[k], P.steps[k], "conv_exp_series", s, 0, pairs));
  ORTH_HIP(launch_tap_items(2, reinterpret_cast<const TapItem*>(ws + P.off_scatter), (int)P.scatter.size(), dtype,
                            P.max_scatter, s));
  return ORTH_OK;
}

int orth_build_conv_kernel(const void* rko, const void* proj, int32_t cin, int32_t cout, int32_t k, int32_t stride,
                           int32_t dilation, int32_t groups, int32_t dtype, void* kernel_out, void* workspace,
                           size_t workspace_bytes, void* stream) {
  orth_conv_desc d;
  d.geom = orth_conv_geom{cin, cout, k, stride, dilation, groups};
  d.rko = rko;
  d.proj = proj;
  d.kernel = kernel_out;
  return orth_build_conv_kernels_batched(&d, 1, dtype, workspace, workspace_bytes, stream);
}

// --------------------------------------------------------------- checks --
namespace {
int validate_check(const orth_check_args* a) {
  if (!a) return fail(ORTH_EINVAL, "args is NULL");
  if (a->mode == ORTH_CHECK_GRAM) {
    if (a->n_mats < 0 || (a->n_mats > 0 && !a->mats)) return fail(ORTH_EINVAL, "bad matrix list");
    if (a->mat_dtype != ORTH_F32 && a->mat_dtype != ORTH_BF16) return fail(ORTH_EINVAL, "unknown dtype");
    for (int i = 0; i < a->n_mats; ++i) {
      const orth_mat& m = a->mats[i];
      if (!m.in || m.rows < 1 || m.cols < 1 || m.ld_in < m.cols || m.rows > (1 << 20) || m.cols > (1 << 20))
        return fail(ORTH_EINVAL, "bad matrix in check list");
    }
    return ORTH_OK;
  }
  if (a->mode != ORTH_CHECK_CONV && a->mode != ORTH_CHECK_CONV_ADJOINT) return fail(ORTH_EINVAL, "unknown check mode");
  int rc = validate_geom(&a->geom);
  if (rc) return rc;
  if (a->kernel_dtype != ORTH_F32 && a->kernel_dtype != ORTH_BF16) return fail(ORTH_EINVAL, "unknown dtype");
  if (!a->kernel || !a->x) return fail(ORTH_EINVAL, "NULL kernel or input");
  if (a->batch < 1 || a->height < 1 || a->width < 1) return fail(ORTH_EINVAL, "batch, height, width must be >= 1");
  if (a->mode == ORTH_CHECK_CONV && (a->height % a->geom.stride || a->width % a->geom.stride))
    return fail(ORTH_EINVAL, "height and width must be divisible by the stride");
  if ((int64_t)a->geom.cout * a->height * a->width * a->geom.stride * a->geom.stride > (int64_t)1 << 31 ||
      (int64_t)a->geom.cin * a->height * a->width * a->geom.stride * a->geom.stride > (int64_t)1 << 31)
    return fail(ORTH_EINVAL, "conv check input too large");
  return ORTH_OK;
}

void gram_check_items(const orth_check_args* a, float* out, GemmList& items) {
  for (int i = 0; i < a->n_mats; ++i) {
    const orth_mat& m = a->mats[i];
    const bool tall = m.rows >= m.cols;
    const int nsz = tall ? m.cols : m.rows, ksz = tall ? m.rows : m.cols;
    const int t = (nsz + 63) / 64;
    for (int ti = 0; ti < t; ++ti)
      for (int tj = 0; tj < t; ++tj) {
        GemmItem g{};
        g.A = g.B = m.in;
        g.lda = g.ldb = m.ld_in;
        g.M = g.N = nsz;
        g.K = ksz;
        g.ti = ti;
        g.tj = tj;
        g.a_dtype = g.b_dtype = a->mat_dtype;
        g.a_trans = g.b_trans = tall ? 1 : 0;
        g.epi = EPI_MAXDEV;
        g.red = out + i;
        items.push_back(g);
      }
  }
}

size_t conv_partial_doubles(const orth_check_args* a) {
  const int s = a->geom.stride;
  int64_t in_ps, out_ps;
  if (a->mode == ORTH_CHECK_CONV) {
    in_ps = (int64_t)a->geom.cin * a->height * a->width;
    out_ps = (int64_t)a->geom.cout * (a->height / s) * (a->width / s);
  } else {
    in_ps = (int64_t)a->geom.cout * a->height * a->width;
    out_ps = (int64_t)a->geom.cin * a->height * s * a->width * s;
  }
  return (size_t)a->batch * (size_t)((in_ps + 255) / 256 + (out_ps + 255) / 256);
}
}  // namespace

int orth_check_workspace_size(const orth_check_args* args, size_t* bytes) {
  if (!bytes) return fail(ORTH_EINVAL, "bytes is NULL");
  int rc = validate_check(args);
  if (rc) return rc;
  if (args->mode == ORTH_CHECK_GRAM) {
    GemmList items;
    gram_check_items(args, nullptr, items);
    *bytes = GemmList::bound(items.size());
  } else {
    *bytes = align_up(sizeof(double) * conv_partial_doubles(args));
  }
  return ORTH_OK;
}

int orth_check_norm(const orth_check_args* args, float* out_dev, void* workspace, size_t workspace_bytes,
                    void* stream) {
  int rc = validate_check(args);
  if (rc) return rc;
  if (!out_dev) return fail(ORTH_EINVAL, "out_dev is NULL");
  size_t need = 0;
  orth_check_workspace_size(args, &need);
  rc = check_workspace(workspace, workspace_bytes, need);
  if (rc) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (args->mode == ORTH_CHECK_GRAM) {
    if (args->n_mats == 0) return ORTH_OK;
    GemmList items;
    gram_check_items(args, out_dev, items);
    TableImage img;
    put(img, 0, items);
    ORTH_HIP(launch_fill_f32(out_dev, args->n_mats, 0.f, s));
    rc = upload_tables(img, workspace, s);
    if (rc) return rc;
    ORTH_HIP(launch_list(static_cast<const unsigned char*>(workspace), 0, items, "check_gram", s));
    return ORTH_OK;
  }
  ORTH_HIP(launch_conv_check(args, args->kernel, args->x, static_cast<double*>(workspace), out_dev,
                             args->mode == ORTH_CHECK_CONV_ADJOINT, s));
  return ORTH_OK;
}

// --------------------------------------------------------------- timing --
int orth_timing_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_timing = on != 0;
  return ORTH_OK;
}

int orth_timing_reset(void) {
  std::lock_guard<std::mutex> lk(g_tmu);
  const int rc = drain_timing_locked();
  g_totals.clear();
  g_spans.clear();
  if (g_ref) g_event_pool.push_back(g_ref);
  g_ref = nullptr;
  return rc ? drain_failed(rc) : ORTH_OK;
}

int orth_timing_read(const char* kernel_name, double* total_ms, int64_t* launches) {
  if (!kernel_name || !total_ms || !launches) return fail(ORTH_EINVAL, "NULL argument");
  std::lock_guard<std::mutex> lk(g_tmu);
  const int rc = drain_timing_locked();
  auto it = g_totals.find(kernel_name);
  *total_ms = it == g_totals.end() ? 0.0 : it->second.first;
  *launches = it == g_totals.end() ? 0 : it->second.second;
  return rc ? drain_failed(rc) : ORTH_OK;
}

int orth_timing_filter(const char* prefixes) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_filter = split_prefixes(prefixes);
  return ORTH_OK;
}

int orth_timing_span(const char* prefixes, double* covered_ms, int64_t* launches) {
  if (!prefixes || !covered_ms || !launches) return fail(ORTH_EINVAL, "NULL argument");
  const std::vector<std::string> pre = split_prefixes(prefixes);
  std::lock_guard<std::mutex> lk(g_tmu);
  const int rc = drain_timing_locked();
  std::vector<std::pair<double, double>> iv;
  for (const auto& kv : g_spans)
    for (const auto& p : pre)
      if (kv.first.compare(0, p.size(), p) == 0) {
        iv.insert(iv.end(), kv.second.begin(), kv.second.end());
        break;
      }
  std::sort(iv.begin(), iv.end());
  double covered = 0.0, lo = 0.0, hi = 0.0;
  for (size_t i = 0; i < iv.size(); ++i) {
    if (i == 0 || iv[i].first > hi) {
      covered += hi - lo;
      lo = iv[i].first;
      hi = iv[i].second;
    } else {
      hi = std::max(hi, iv[i].second);
    }
  }
  if (!iv.empty()) covered += hi - lo;
  *covered_ms = covered;
  *launches = (int64_t)iv.size();
  return rc ? drain_failed(rc) : ORTH_OK;
}

int orth_timing_names(char* buf, size_t buf_bytes) {
  if (!buf || buf_bytes == 0) return fail(ORTH_EINVAL, "NULL buffer");
  std::lock_guard<std::mutex> lk(g_tmu);
  const int rc = drain_timing_locked();
  if (rc) return drain_failed(rc);
  std::string all;
  for (auto& kv : g_totals) {
    if (!all.empty()) all += ";";
    all += kv.first;
  }
  if (all.size() + 1 > buf_bytes) return fail(ORTH_EINVAL, "buffer too small");
  std::memcpy(buf, all.c_str(), all.size() + 1);
  return ORTH_OK;
}

}  // extern "C"
