// CPU stand-ins for the HIP runtime calls and kernel launchers that the
// library's host code (csrc/host.hip) makes, so that the planner, the
// validation, the workspace layout and the descriptor uploads run on a
// machine without a GPU under AddressSanitizer and UndefinedBehaviorSanitizer.
//
// "Device" memory is address space reserved with PROT_NONE: nothing may
// dereference it on the host (a stray access faults).  Copies into it are
// checked and recorded instead of performed: the destination must lie in a
// registered device range, the host source is read in full (so that the
// sanitizer checks the whole source), and the written byte ranges are kept.
// Every launcher then checks that the descriptor tables it is handed lie
// inside registered device memory and were written by a copy since the last
// stub_reset() on the same thread — i.e. that a call uploads every table
// byte its launches read.  A violation prints its kind and aborts.  The
// stand-ins are safe to call from several threads at once.
#include <sys/mman.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <iterator>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../paper_2601_13776_amd/csrc/internal.h"

// log2 of the reserved "device" address space (32 TiB by default; the
// ThreadSanitizer build takes less, to fit its application ranges)
#ifndef STUB_ARENA_BITS
#define STUB_ARENA_BITS 45
#endif

namespace {
std::mutex g_mu;
std::map<uintptr_t, uintptr_t> g_dev;       // registered device ranges [begin, end)
// written ranges since the calling thread's last reset, merged: a call's
// copies and launches all happen on the thread that made the call
thread_local std::map<uintptr_t, uintptr_t> g_written;
long g_launches = 0;
thread_local long t_launches = 0;           // launches of the calling thread
long g_copies = 0;
unsigned char* g_arena = nullptr;           // reserved PROT_NONE address space
size_t g_arena_size = 0, g_arena_used = 0;

[[noreturn]] void violation(const char* what, const char* where, uintptr_t p, size_t n) {
  std::fprintf(stderr, "STUB VIOLATION: %s in %s at %#lx (+%zu bytes)\n", what, where, (unsigned long)p, n);
  std::fflush(stderr);
  std::abort();
}

bool in_device(uintptr_t p, size_t n) {
  auto it = g_dev.upper_bound(p);
  if (it == g_dev.begin()) return false;
  --it;
  return p >= it->first && p + n <= it->second;
}

bool covered(uintptr_t p, size_t n) {
  if (n == 0) return true;
  auto it = g_written.upper_bound(p);
  if (it == g_written.begin()) return false;
  --it;
  return p >= it->first && p + n <= it->second;
}

void mark_written(uintptr_t p, size_t n) {
  if (n == 0) return;
  uintptr_t b = p, e = p + n;
  auto it = g_written.upper_bound(b);
  if (it != g_written.begin()) {
    auto prev = std::prev(it);
    if (prev->second >= b) {
      b = prev->first;
      e = std::max(e, prev->second);
      it = g_written.erase(prev);
    }
  }
  while (it != g_written.end() && it->first <= e) {
    e = std::max(e, it->second);
    it = g_written.erase(it);
  }
  g_written[b] = e;
}

// a descriptor table of `n` elements of T read by a launch
template <typename T>
void table(const T* p, long n, const char* where) {
  if (n <= 0) return;
  std::lock_guard<std::mutex> lk(g_mu);
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  const size_t bytes = sizeof(T) * (size_t)n;
  if (!in_device(a, bytes)) violation("table outside device memory", where, a, bytes);
  if (!covered(a, bytes)) violation("table not uploaded by this call", where, a, bytes);
}

#ifdef PLANT_RACE
long g_racy = 0;   // a counter every thread bumps without the lock: a planted race
#endif

hipError_t launched() {
#ifdef PLANT_RACE
  ++g_racy;
#endif
  std::lock_guard<std::mutex> lk(g_mu);
  ++g_launches;
  ++t_launches;
  return hipSuccess;
}
}  // namespace

// ------------------------------------------------------------ stub API ----
extern "C" {

// Fake device allocation: bytes rounded to 256, from PROT_NONE space.
void* stub_dev_alloc(size_t bytes) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_arena) {
    g_arena_size = (size_t)1 << STUB_ARENA_BITS;   // address space only, nothing committed
    void* p = mmap(nullptr, g_arena_size, PROT_NONE, MAP_PRIVATE | MAP_ANONYMOUS | MAP_NORESERVE, -1, 0);
    if (p == MAP_FAILED) {
      std::fprintf(stderr, "stub: cannot reserve device address space\n");
      std::abort();
    }
    g_arena = static_cast<unsigned char*>(p);
  }
  bytes = (bytes + 255) / 256 * 256;
  if (bytes == 0) bytes = 256;
  if (g_arena_used + bytes + 4096 > g_arena_size) {
    std::fprintf(stderr, "stub: device address space exhausted\n");
    std::abort();
  }
  unsigned char* p = g_arena + g_arena_used;
  g_arena_used += bytes + 4096;   // a guard gap after every allocation
  g_dev[reinterpret_cast<uintptr_t>(p)] = reinterpret_cast<uintptr_t>(p) + bytes;
  return p;
}

void stub_reset(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_written.clear();
}

long stub_launches(void) { return t_launches; }

long stub_launches_total(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  return g_launches;
}

// Checks of the checks: 0 launches from a table no copy wrote, 1 copies
// outside device memory; each must end the process with a violation.
void stub_selftest(int which) {
  unsigned char* d = static_cast<unsigned char*>(stub_dev_alloc(4096));
  if (which == 0) {
    int v = 0;
    hipMemcpyAsync(d, &v, sizeof v, hipMemcpyHostToDevice, nullptr);
    table(reinterpret_cast<const int*>(d), 2, "selftest");     // the second element was never written
  } else {
    int v = 0;
    hipMemcpyAsync(d + 4093, &v, sizeof v, hipMemcpyHostToDevice, nullptr);   // runs past the allocation
  }
}

long stub_copies(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  return g_copies;
}

// ------------------------------------------------------- HIP runtime ----
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind kind, hipStream_t) {
  std::lock_guard<std::mutex> lk(g_mu);
  ++g_copies;
  const uintptr_t d = reinterpret_cast<uintptr_t>(dst), s = reinterpret_cast<uintptr_t>(src);
  if (!in_device(d, bytes)) violation("copy destination outside device memory", "hipMemcpyAsync", d, bytes);
  if (kind == hipMemcpyHostToDevice) {
    // read every source byte: the sanitizer checks the host image
    volatile unsigned char sink = 0;
    const unsigned char* h = static_cast<const unsigned char*>(src);
    for (size_t i = 0; i < bytes; ++i) sink ^= h[i];
    (void)sink;
  } else if (kind == hipMemcpyDeviceToDevice) {
    if (!in_device(s, bytes)) violation("copy source outside device memory", "hipMemcpyAsync", s, bytes);
  } else {
    violation("unexpected copy kind", "hipMemcpyAsync", d, bytes);
  }
  mark_written(d, bytes);
  return hipSuccess;
}

// Pinned buffers are real host memory (the library writes its table images
// there).  The library keeps them for the life of the process, as it does
// on a GPU; the registry keeps them reachable for the leak checker.
std::vector<void*>* host_allocs() {
  static auto* v = new std::vector<void*>();
  return v;
}
hipError_t hipHostMalloc(void** p, size_t bytes, unsigned int) {
  *p = std::malloc(bytes);
  if (!*p) return hipErrorOutOfMemory;
  std::lock_guard<std::mutex> lk(g_mu);
  host_allocs()->push_back(*p);
  return hipSuccess;
}
hipError_t hipHostFree(void* p) {
  std::lock_guard<std::mutex> lk(g_mu);
  auto* v = host_allocs();
  for (auto it = v->begin(); it != v->end(); ++it)
    if (*it == p) {
      v->erase(it);
      std::free(p);
      return hipSuccess;
    }
  violation("free of memory not from hipHostMalloc", "hipHostFree", reinterpret_cast<uintptr_t>(p), 0);
}

// Events and streams are opaque handles that nothing dereferences.
int g_handle;
hipError_t hipEventCreate(hipEvent_t* e) {
  *e = reinterpret_cast<hipEvent_t>(&g_handle);
  return hipSuccess;
}
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }
hipError_t hipEventQuery(hipEvent_t) { return hipSuccess; }
hipError_t hipEventSynchronize(hipEvent_t) { return hipSuccess; }
hipError_t hipEventElapsedTime(float* ms, hipEvent_t, hipEvent_t) {
  *ms = 0.f;
  return hipSuccess;
}
hipError_t hipStreamCreateWithFlags(hipStream_t* s, unsigned) {
  *s = reinterpret_cast<hipStream_t>(&g_handle);
  return hipSuccess;
}
hipError_t hipStreamWaitEvent(hipStream_t, hipEvent_t, unsigned) { return hipSuccess; }
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
hipError_t hipStreamGetDevice(hipStream_t, hipDevice_t* d) {
  *d = 0;
  return hipSuccess;
}
hipError_t hipStreamIsCapturing(hipStream_t, hipStreamCaptureStatus* c) {
  *c = hipStreamCaptureStatusNone;
  return hipSuccess;
}
hipError_t hipGetDevice(int* d) {
  *d = 0;
  return hipSuccess;
}
hipError_t hipSetDevice(int) { return hipSuccess; }
hipError_t hipPeekAtLastError(void) { return hipSuccess; }
const char* hipGetErrorString(hipError_t) { return "hip stub"; }

}  // extern "C"

// ----------------------------------------------------------- launchers ----
namespace orth {

hipError_t launch_bjorck_small(const SmallMat* mats, int n, int, int, int, float, int, int, int, int, int32_t*,
                               hipStream_t) {
  table(mats, n, "launch_bjorck_small");
  return launched();
}
hipError_t launch_bjorck_small_vjp(const SmallVjpMat* mats, int n, int, int, int, float, int, int, int, int, int32_t*,
                                   hipStream_t) {
  table(mats, n, "launch_bjorck_small_vjp");
  return launched();
}
hipError_t launch_power_init(const TiledMat* mats, int n, hipStream_t) {
  table(mats, n, "launch_power_init");
  return launched();
}
hipError_t launch_power_keep(const TiledMat* mats, int n, int, hipStream_t) {
  table(mats, n, "launch_power_keep");
  return launched();
}
hipError_t launch_spec_bwd(const TiledMat* mats, const TiledMat* bw, int n, const PowerItem* i0, int n0,
                           const PowerItem* i1, int n1, int, int, const int32_t*, hipStream_t) {
  table(mats, n, "launch_spec_bwd (mats)");
  table(bw, n, "launch_spec_bwd (backward table)");
  table(i0, n0, "launch_spec_bwd (X products)");
  table(i1, n1, "launch_spec_bwd (X^T products)");
  return launched();
}
hipError_t launch_power_dot(const TiledMat*, const PowerItem* items, int n, int, hipStream_t) {
  table(items, n, "launch_power_dot");
  return launched();
}
hipError_t launch_power_normalize(const TiledMat* mats, int n, hipStream_t) {
  table(mats, n, "launch_power_normalize");
  return launched();
}
hipError_t launch_prescale_partial(const TiledMat*, const TileItem* items, int n, int, double*, hipStream_t) {
  table(items, n, "launch_prescale_partial");
  return launched();
}
hipError_t launch_prescale_finish(const TiledMat* mats, int n, const double*, int, int32_t*, hipStream_t, int) {
  table(mats, n, "launch_prescale_finish");
  return launched();
}
hipError_t launch_prescale_scale(const TiledMat*, const TileItem* items, int n, int, int, hipStream_t) {
  table(items, n, "launch_prescale_scale");
  return launched();
}
hipError_t launch_writeout(const TiledMat*, const TileItem* items, int n, int, int, hipStream_t) {
  table(items, n, "launch_writeout");
  return launched();
}
hipError_t launch_bf16_tiles(int, const TiledMat*, const TileItem* items, int n, float, hipStream_t, int, int) {
  table(items, n, "launch_bf16_tiles");
  return launched();
}
hipError_t launch_gemm_f32(const GemmItem* items, const GemmTile* tiles, int n_tiles, const char* name, hipStream_t,
                           int, const GemmPair*, int n_km) {
  if (n_km < 0 || n_km > n_tiles) violation("k-major tile count out of range", name, 0, (size_t)n_km);
  if (n_tiles > 0) table(items, 1, name);
  table(tiles, n_tiles, name);
  return launched();
}
hipError_t launch_vjp_load_grad(const TiledMat*, const TileItem* items, int n, int, hipStream_t) {
  table(items, n, "launch_vjp_load_grad");
  return launched();
}
hipError_t launch_vjp_dot_partial(const TiledMat*, const TileItem* items, int n, int, double*, hipStream_t) {
  table(items, n, "launch_vjp_dot_partial");
  return launched();
}
hipError_t launch_vjp_dot_finish(const TiledMat* mats, int n, const double*, hipStream_t) {
  table(mats, n, "launch_vjp_dot_finish");
  return launched();
}
hipError_t launch_vjp_writeout(const TiledMat*, const TileItem* items, int n, int, int, const int32_t*, hipStream_t) {
  table(items, n, "launch_vjp_writeout");
  return launched();
}
hipError_t launch_compose_init(const ComposeGroup* groups, int n, int, int64_t, hipStream_t) {
  table(groups, n, "launch_compose_init");
  return launched();
}
hipError_t launch_compose_combine(const ComposeGroup*, const CombineItem* items, int n, int64_t, hipStream_t) {
  table(items, n, "launch_compose_combine");
  return launched();
}
hipError_t launch_fill_f32(float*, int64_t, float, hipStream_t) { return launched(); }
hipError_t launch_tap_items(int, const TapItem* items, int n, int, int64_t, hipStream_t, const char*) {
  table(items, n, "launch_tap_items");
  return launched();
}
hipError_t launch_exp_skew(const ExpItem* items, int n, int, int, int64_t, hipStream_t) {
  table(items, n, "launch_exp_skew");
  return launched();
}
hipError_t launch_exp_init(const ExpItem* items, int n, int, int64_t, hipStream_t) {
  table(items, n, "launch_exp_init");
  return launched();
}
hipError_t launch_conv_apply(const orth_conv_apply_args*, hipStream_t) { return launched(); }
hipError_t launch_conv_check(const orth_check_args*, const void*, const float*, double*, float*, int, hipStream_t) {
  return launched();
}

}  // namespace orth
