// bench_read.hip -- streaming-read ceiling of the GPU, for the benchmark's report only (not
// part of libsdblock.so): how fast plain 16-byte loads can read a buffer that no cache holds.
// Built into libsdbench.so.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef unsigned v4u32 __attribute__((ext_vector_type(4)));

// Workgroup b reads bytes [b * per, (b + 1) * per) of the buffer (per a multiple of 16), 8
// non-temporal 16-byte loads per thread in flight; the loaded words are folded into one
// value that is stored only if it equals `magic`, a value the compiler cannot know, so no
// load can be dropped (a store of one word, if the data ever fold to it, is harmless).
__global__ __launch_bounds__(512) void stream_read_kernel(const char *buf, unsigned long long per, unsigned magic,
                                                          unsigned *sink) {
  const v4u32 *p = reinterpret_cast<const v4u32 *>(buf + (unsigned long long)blockIdx.x * per);
  const unsigned n = (unsigned)(per / 16);
  v4u32 acc = {0u, 0u, 0u, 0u};
  unsigned i = threadIdx.x;
  for (; i + 7u * 512u < n; i += 8u * 512u) {
    v4u32 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(p + i + 512u * u);
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= v[u];
  }
  for (; i < n; i += 512u) acc ^= __builtin_nontemporal_load(p + i);
  const unsigned x = acc.x ^ acc.y ^ acc.z ^ acc.w;
  if (x == magic) sink[blockIdx.x] = x;
}

extern "C" {

// Read `bytes` of device memory at `buf` with `grid` workgroups of 512 threads on `stream`.
// bytes must be a multiple of 16 * grid; sink holds `grid` words (never written in practice).
// Returns 0, or -1 on a bad argument, or the HIP error code of the launch.
int sdbench_stream_read(const void *buf, unsigned long long bytes, int grid, unsigned *sink, void *stream) {
  if (!buf || !sink || grid < 1 || bytes == 0 || bytes % (16ull * (unsigned)grid)) return -1;
  const unsigned long long per = bytes / (unsigned)grid;
  if (per / 16 > 0xffffffffull) return -1;
  hipLaunchKernelGGL(stream_read_kernel, dim3(grid), dim3(512), 0, (hipStream_t)stream, (const char *)buf, per, 0x9e3779b9u,
                     sink);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // extern "C"
