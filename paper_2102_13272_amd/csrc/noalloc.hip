// nwg_conv2d_noalloc: the convolution of nwg_conv2d for callers that cannot
// allocate device memory (code under stream capture, serving loops,
// harnesses that forbid hipMalloc).  Its workspace is one static device
// array per GPU; it calls no hipMalloc, hipFree or allocating routine.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "nwg_internal.h"

namespace {

// The workspace of every nwg_conv2d_noalloc call on a GPU: U, V and Z (with
// the partial sums or scratch the plan's layout puts after Z), each at a
// 256-byte boundary.  Each device holds its own copy of the array, from the
// first launch of this library's code on it until the process ends.  Host
// code never passes `scratch` itself to a kernel (in host code the name is
// a stand-in, not a device address): it takes the device's address from
// hipGetSymbolAddress once per device and passes that.
static __device__ __align__(256) unsigned char scratch[NWG_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
unsigned char* g_scratch_ptr[kMaxDevices];   // per device, NULL until resolved

// The current device's scratch address, resolved on its first call (with
// that device current) and kept.
int scratch_of_current_device(unsigned char** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    hipGetLastError();
    return nwg::fail(NWG_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  }
  if (dev < 0 || dev >= kMaxDevices)
    return nwg::fail(NWG_EUNSUPPORTED, "device %d: the static scratch serves devices 0..%d", dev,
                     kMaxDevices - 1);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      hipGetLastError();
      return nwg::fail(NWG_EHIP, "hipGetSymbolAddress of the static scratch on device %d: %s",
                       dev, hipGetErrorString(e));
    }
    g_scratch_ptr[dev] = static_cast<unsigned char*>(ptr);
  }
  *out = g_scratch_ptr[dev];
  return NWG_OK;
}

constexpr size_t round256(size_t b) { return (b + 255) & ~(size_t)255; }

}  // namespace

extern "C" int nwg_conv2d_noalloc(int B, int M, int N, int H, int W, int r, int pad, int tile,
                                  const float* x, const float* w, float* y, void* stream) {
  if (!x || !w || !y) return nwg::fail(NWG_EINVAL, "NULL argument to nwg_conv2d_noalloc");
  nwg_plan_info g;
  int rc = nwg::compute_geometry(B, M, N, H, W, r, pad, tile, 0, &g);
  if (rc != NWG_OK) return rc;
  rc = nwg::check_plan_request(g);
  if (rc != NWG_OK) return rc;
  const size_t ub = g.u_bytes;
  const size_t vb = nwg::plan_holds_v(g) ? g.v_bytes : 0;
  const size_t zb = nwg::plan_holds_z(g) ? nwg::zalloc_bytes(g) : 0;
  const size_t need = round256(ub) + round256(vb) + round256(zb);
  if (need > NWG_NOALLOC_SCRATCH_BYTES)
    return nwg::fail(NWG_EUNSUPPORTED,
                     "workspace of %zu bytes exceeds the static scratch of %zu bytes", need,
                     (size_t)NWG_NOALLOC_SCRATCH_BYTES);
  if ((((uintptr_t)x | (uintptr_t)w | (uintptr_t)y) & 15) != 0)
    return nwg::fail(NWG_EINVAL, "x, w and y must be 16-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (s) {
    // the scratch is the current device's: the stream must run there
    int sdev = -1, cur = -1;
    if (hipStreamGetDevice(s, &sdev) != hipSuccess || hipGetDevice(&cur) != hipSuccess) {
      hipGetLastError();
      return nwg::fail(NWG_EHIP, "device of the stream or current device unknown");
    }
    if (sdev != cur)
      return nwg::fail(NWG_EINVAL, "the stream runs on device %d, device %d is current", sdev,
                       cur);
  }
  unsigned char* base = nullptr;
  rc = scratch_of_current_device(&base);
  if (rc != NWG_OK) return rc;
  // nothing here needs to start at zero: every kernel writes each value of
  // U, V and Z it later reads
  float* U = ub ? reinterpret_cast<float*>(base) : nullptr;
  float* V = vb ? reinterpret_cast<float*>(base + round256(ub)) : nullptr;
  float* Z = zb ? reinterpret_cast<float*>(base + round256(ub) + round256(vb)) : nullptr;
  rc = nwg::kernel_transform_into(g, w, U, s);
  if (rc != NWG_OK) return rc;
  return nwg::conv_steps(g, U, V, Z, x, y, s);
}
