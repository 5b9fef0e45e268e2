// Achievable read bandwidth of a device buffer, for the bench's context figure: the
// same-run time of a plain streaming read of the frames buffer (no hashing, no table),
// beside which the algorithmic HBM figures of the tree-building kernels are reported.
// Not part of the library's call-path API (include/cct.h); bench.py loads it on its own.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kThreads = 768;       // 12 waves per workgroup, one workgroup per CU
constexpr int64_t kTile = 8192;     // bytes per wave and iteration: eight 1 KiB coalesced loads

// Tiles of 8 KiB are dealt to the waves round-robin, so the whole grid sweeps memory in
// order; every lane reads 16 bytes of each 1 KiB row with the same 16-byte raw buffer
// load the ingest kernel streams its frames with (a wave-uniform descriptor per tile,
// so the descriptor stays in scalar registers).  The xor of the data is kept so the
// loads stay live; one word per workgroup is written only if it matches a value the
// data cannot produce by chance in this use.
__global__ __launch_bounds__(kThreads) void read_kernel(const unsigned char *p, int64_t bytes, uint32_t *sink) {
  const int lane = threadIdx.x & 63;
  const int64_t waves = (int64_t)gridDim.x * (kThreads / 64);
  const int64_t w = __builtin_amdgcn_readfirstlane((int)(blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6)));
  const int64_t tiles = bytes / kTile;
  uint32_t acc = 0;
  for (int64_t t = w; t < tiles; t += waves) {
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc((void *)(p + t * kTile), (short)0, (int)kTile, 0x00020000);
    u32x4 v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = __builtin_amdgcn_raw_buffer_load_b128(r, 16 * lane + 1024 * k, 0, 0);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc ^= v[k][0] ^ v[k][1] ^ v[k][2] ^ v[k][3];
  }
  const u32x4 *q = (const u32x4 *)p;
  for (int64_t i = tiles * (kTile / 16) + w * 64 + lane; i < bytes / 16; i += waves * 64) {
    const u32x4 v = q[i];
    acc ^= v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  if (acc == 0x9E3779B9u) sink[blockIdx.x] = acc;
}

}  // namespace

extern "C" {

// Best time of `reps` reads of `bytes` bytes (rounded down to 16) at the 16-byte aligned
// device address p, on `stream`; sink is device memory of at least one word per CU.
// Returns 0, or -1 on a bad argument or a failed HIP call.
int cctbw_read(const void *p, int64_t bytes, uint32_t *sink, void *stream, int reps, float *best_ms) {
  if (!p || !sink || !best_ms || bytes < 16 || reps < 1 || ((uintptr_t)p & 15)) return -1;
  hipStream_t s = (hipStream_t)stream;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return -1;
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess) return -1;
  if (hipEventCreate(&e1) != hipSuccess) { (void)hipEventDestroy(e0); return -1; }
  float best = 1e30f;
  int rc = 0;
  for (int r = 0; r < reps && rc == 0; ++r) {
    float ms = 0;
    if (hipEventRecord(e0, s) != hipSuccess) { rc = -1; break; }
    hipLaunchKernelGGL(read_kernel, dim3(cus), dim3(kThreads), 0, s, (const unsigned char *)p, bytes, sink);
    if (hipGetLastError() != hipSuccess || hipEventRecord(e1, s) != hipSuccess ||
        hipEventSynchronize(e1) != hipSuccess || hipEventElapsedTime(&ms, e0, e1) != hipSuccess) {
      rc = -1;
      break;
    }
    if (ms < best) best = ms;
  }
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (rc == 0) *best_ms = best;
  return rc;
}

}  // extern "C"
