// Finite check of a call's floating-point inputs: a debugging aid that
// map_set_finite_check switches on (off by default).  Each launch scans one
// buffer with a grid-stride loop (32-bit words; bf16: two values per word
// when the buffer is 4-byte aligned) and raises a device flag if any value
// has an all-ones exponent (an infinity or a NaN); several launches may
// raise the same flag.
#include "internal.h"

namespace mapk {

namespace {

// The flag the scans raise (one per device; the host clears and reads it).
__device__ int g_nonfinite;

// mode 0: float32 words; 1: bfloat16 pairs in 32-bit words; 2: bfloat16
// values one by one (a buffer not 4-byte aligned)
__global__ __launch_bounds__(256) void finite_kernel(const void* p, long long n, int mode, const uint16_t* tail,
                                                     int* flag) {
  int bad = 0;
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long i = static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
    if (mode == 2) {
      const uint32_t u = static_cast<const uint16_t*>(p)[i];
      bad |= (u & 0x7f80u) == 0x7f80u;
    } else {
      const uint32_t u = static_cast<const uint32_t*>(p)[i];
      bad |= mode ? ((u & 0x7f80u) == 0x7f80u) | ((u & 0x7f800000u) == 0x7f800000u)
                  : (u & 0x7f800000u) == 0x7f800000u;
    }
  }
  if (tail && blockIdx.x == 0 && threadIdx.x == 0) bad |= (*tail & 0x7f80u) == 0x7f80u;  // odd bf16 count
  if (bad) *flag = 1;
}

}  // namespace

int* finite_flag() {
  static int* addr[16] = {nullptr};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 16) return nullptr;
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(g_nonfinite)) != hipSuccess) return nullptr;
    addr[dev] = static_cast<int*>(p);
  }
  return addr[dev];
}

hipError_t launch_finite_check(const void* p, long long count, int elem_bytes, int* flag, hipStream_t s) {
  if (!p || count <= 0) return hipSuccess;
  int mode = elem_bytes == 2 ? 1 : 0;
  long long n = count;
  const uint16_t* tail = nullptr;
  if (mode == 1) {
    if (reinterpret_cast<uintptr_t>(p) & 3) {
      mode = 2;  // element by element
    } else {
      n = count / 2;
      if (count & 1) tail = static_cast<const uint16_t*>(p) + (count - 1);
    }
  }
  const long long want = (n + 255) / 256;
  const int blocks = static_cast<int>(want < 1 ? 1 : (want > 4096 ? 4096 : want));
  return launch_kernel("finite_check", finite_kernel, dim3(blocks), dim3(256), 0, s, p, n, mode, tail, flag);
}

}  // namespace mapk
