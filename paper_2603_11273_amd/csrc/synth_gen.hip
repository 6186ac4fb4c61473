// Seeded input generator on the device (libasr_synth.so).
//
// Test and benchmark input only: this library holds none of the step's
// arithmetic.  It evaluates the counter-based generator that the Python
// module synth.py defines (value i of a stream is a function of
// (seed, stream, i) alone) directly in device memory, so full-size weights
// and caches need no host round trip.  The hash is Chris Wellons'
// "lowbias32" integer mixer from his hash-prospector project; a value is
//   h = lowbias32((lowbias32(i ^ k1) + k2) mod 2^32),
//   k = floor(h * levels / 2^32) - kmax,   x = k * 2^-bits + offset,
// and, for the "fine" variant whose values bf16 cannot hold, plus
//   j * 2^-(bits + 10) with j drawn the same way from a second stream
// (|j| <= 255).  Every value is a short binary fraction, exact in float32,
// so the device and the host route agree bit for bit.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

__device__ __forceinline__ uint32_t lowbias32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7FEB352Du;
  x ^= x >> 15;
  x *= 0x846CA68Bu;
  x ^= x >> 16;
  return x;
}

__device__ __forceinline__ int32_t draw(uint32_t i, uint32_t k1, uint32_t k2, uint32_t levels,
                                        int32_t kmax) {
  const uint32_t h = lowbias32(lowbias32(i ^ k1) + k2);
  return (int32_t)(((uint64_t)h * levels) >> 32) - kmax;
}

struct GridArgs {
  float* out;
  int64_t count;
  uint32_t start;      // counter of out[0]; start + count <= 2^32
  uint32_t k1, k2;     // stream keys
  uint32_t levels;     // 2 kmax + 1
  int32_t kmax;
  float scale;         // 2^-bits
  float offset;
  int32_t fine;        // add the second-stream term
  uint32_t f1, f2;     // its stream keys
  float fine_scale;    // 2^-(bits + 10)
};

__global__ void k_grid(GridArgs a) {
  const int64_t step = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < a.count; i += step) {
    const uint32_t c = a.start + (uint32_t)i;
    float v = (float)draw(c, a.k1, a.k2, a.levels, a.kmax) * a.scale;
    if (a.offset != 0.0f) v = v + a.offset;
    if (a.fine) v = v + (float)draw(c, a.f1, a.f2, 511u, 255) * a.fine_scale;
    a.out[i] = v;
  }
}

}  // namespace

extern "C" {

// Fills out[0 .. count) (device memory) on `stream`; returns 0, or -1 for a
// bad argument, or the HIP error code of the launch.
int asr_synth_grid(float* out, int64_t count, uint32_t start, uint32_t k1, uint32_t k2,
                   int32_t kmax, int32_t bits, float offset, int32_t fine, uint32_t f1,
                   uint32_t f2, void* stream) {
  if (!out || count < 0 || kmax <= 0 || kmax > 255 || bits < 0 || bits > 100) return -1;
  if ((uint64_t)start + (uint64_t)count > (1ull << 32)) return -1;
  if (count == 0) return 0;
  GridArgs a;
  a.out = out;
  a.count = count;
  a.start = start;
  a.k1 = k1;
  a.k2 = k2;
  a.levels = 2u * (uint32_t)kmax + 1u;
  a.kmax = kmax;
  a.scale = ldexpf(1.0f, -bits);
  a.offset = offset;
  a.fine = fine;
  a.f1 = f1;
  a.f2 = f2;
  a.fine_scale = ldexpf(1.0f, -(bits + 10));
  int64_t blocks = (count + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_grid, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, a);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : (int)e;
}

}  // extern "C"
