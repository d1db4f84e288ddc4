// Plain device-to-device copy of a known size (1 GiB read, 1 GiB written per
// launch, three launches), run under rocprofv3 to scale the FETCH_SIZE and
// WRITE_SIZE counters (KiB per dispatch) to bytes: factor = 2^30 / counter bytes.
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>

__global__ void copy_1gib(const uint4* __restrict__ a, uint4* __restrict__ b, size_t n16) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x) b[i] = a[i];
}

int main() {
  const size_t bytes = (size_t)1 << 30;
  void *a = nullptr, *b = nullptr;
  if (hipMalloc(&a, bytes) != hipSuccess || hipMalloc(&b, bytes) != hipSuccess) return 1;
  if (hipMemset(a, 1, bytes) != hipSuccess) return 1;
  for (int r = 0; r < 3; ++r) copy_1gib<<<8192, 256>>>((const uint4*)a, (uint4*)b, bytes / 16);
  if (hipDeviceSynchronize() != hipSuccess) return 1;
  printf("copied 3 x 1 GiB\n");
  return 0;
}
