// Allocation-free orthogonalization: orth_orthogonalize_batched with a fixed
// device array of the library in place of the caller's workspace, for
// callers that cannot allocate (tight serving loops, harnesses that forbid
// allocation; not code under HIP graph capture, which it refuses).  The call allocates nothing:
// the scratch below instead of a workspace, descriptor tables copied from
// pageable host memory instead of the pinned staging pool, every kernel on
// the caller's stream instead of side streams.
#include <map>
#include <mutex>
#include <string>

#include "internal.h"

namespace orth {

// The scratch of every allocation-free call on a device.  Each GPU that
// loads the library holds its own copy until the process ends.  On the
// host this name is only a stand-in for the symbol: its device address
// (a different one on every GPU) comes from hipGetSymbolAddress and is the
// only form host code passes on.
static __device__ __align__(256) unsigned char scratch[ORTH_NOALLOC_SCRATCH_BYTES];

namespace {
std::mutex g_scratch_mu;
std::map<int, unsigned char*> g_scratch_ptr;   // device -> address of its scratch

// The device address of `scratch` on device `dev`, looked up once per
// device with that device current (the caller's current device is
// restored).
int scratch_of(int dev, unsigned char** out) {
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  auto it = g_scratch_ptr.find(dev);
  if (it != g_scratch_ptr.end()) {
    *out = it->second;
    return ORTH_OK;
  }
  int cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
  void* p = nullptr;
  if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (cur != dev) {
    const hipError_t r = hipSetDevice(cur);
    if (e == hipSuccess) e = r;
  }
  if (e != hipSuccess || !p)
    return report_error(ORTH_EHIP, (std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e)).c_str());
  g_scratch_ptr[dev] = static_cast<unsigned char*>(p);
  *out = static_cast<unsigned char*>(p);
  return ORTH_OK;
}

// Descriptor tables straight from the planner's host image (pageable
// memory: HIP has read the source when hipMemcpyAsync returns).
int upload_pageable(const unsigned char* data, const std::pair<size_t, size_t>* spans, size_t n_spans, void* dst,
                    hipStream_t s) {
  size_t at = 0;
  for (size_t i = 0; i < n_spans; ++i) {
    const hipError_t e = hipMemcpyAsync(static_cast<unsigned char*>(dst) + spans[i].first, data + at,
                                        spans[i].second, hipMemcpyHostToDevice, s);
    if (e != hipSuccess)
      return report_error(ORTH_EHIP, (std::string("hipMemcpyAsync: ") + hipGetErrorString(e)).c_str());
    at += spans[i].second;
  }
  return ORTH_OK;
}
}  // namespace

}  // namespace orth

extern "C" int orth_orthogonalize_batched_noalloc(const orth_mat* mats, int32_t n, const orth_bjorck_opts* opts,
                                                  int32_t* status_dev, void* stream) {
  using namespace orth;
  // validation and sizing on the host, before the device is touched
  size_t need = 0;
  int rc = orth_orthogonalize_workspace_size(mats, n, opts, &need);
  if (rc) return rc;
  if (n == 0) return ORTH_OK;
  if (need > ORTH_NOALLOC_SCRATCH_BYTES) {
    const std::string msg = "batch needs " + std::to_string(need) +
                            " bytes of scratch; orth_orthogonalize_batched_noalloc holds " +
                            std::to_string((size_t)ORTH_NOALLOC_SCRATCH_BYTES) +
                            " (call orth_orthogonalize_batched with a workspace)";
    return report_error(ORTH_EWORKSPACE, msg.c_str());
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  // A captured call could not be replayed: its table copies read host
  // memory that lives only during the call.
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(s, &cap);
  if (e != hipSuccess)
    return report_error(ORTH_EHIP, (std::string("hipStreamIsCapturing: ") + hipGetErrorString(e)).c_str());
  if (cap != hipStreamCaptureStatusNone)
    return report_error(ORTH_EUNSUPPORTED,
                        "orth_orthogonalize_batched_noalloc cannot be captured into a HIP graph: its descriptor "
                        "tables are copied from host memory that lives only during the call");
  int dev = 0;
  e = s ? hipStreamGetDevice(s, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess)
    return report_error(ORTH_EHIP, (std::string("device of the stream: ") + hipGetErrorString(e)).c_str());
  unsigned char* ws = nullptr;
  rc = scratch_of(dev, &ws);
  if (rc) return rc;
  return ortho_enqueue(mats, n, opts, ws, ORTH_NOALLOC_SCRATCH_BYTES, status_dev, s, false, upload_pageable,
                       "orth_orthogonalize_batched_noalloc");
}
