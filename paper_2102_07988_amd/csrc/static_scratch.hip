// The library's per-device static scratch: a fixed-size array in device
// global memory that tp_slice_forward_static uses for the partial sums of the
// slice's kernels (split-K GEMM partials, key-split attention partials)
// instead of the stage workspace, so that call allocates nothing.
//
// In host code the array's name only stands for the symbol: its device
// address is looked up once per device (with that device current) and kept;
// kernels receive that address.  Each device holds its own copy until the
// process ends.  Calls that share a device share its array.
#include <hip/hip_runtime.h>

#include <mutex>

namespace tp {

constexpr size_t STATIC_SCRATCH_BYTES = (size_t)32 << 20;  // 32 MiB
constexpr int MAX_DEVICES = 64;

static __device__ __align__(256) unsigned char scratch[STATIC_SCRATCH_BYTES];

// Device address of the current device's array (nullptr on a HIP error or a
// device index past MAX_DEVICES); *bytes = its size.
void* static_scratch(size_t* bytes) {
  static std::mutex mu;
  static void* addr[MAX_DEVICES] = {};
  *bytes = STATIC_SCRATCH_BYTES;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    addr[dev] = p;
  }
  return addr[dev];
}

}  // namespace tp
