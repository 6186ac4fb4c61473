// Elementwise and row kernels: fills, conversions, weight packing, LayerNorm,
// decoder embedding, and the log-mel front-end.
#include "asr_device.h"

#include <algorithm>

namespace asr {

// ---------------------------------------------------------------------------
// Fills and conversions
// ---------------------------------------------------------------------------
__global__ void k_fill_u32(uint32_t* p, uint32_t v, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}
__global__ void k_fill_f32(float* p, float v, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

static int grid_for(int64_t n, int block = 256) {
  int64_t g = (n + block - 1) / block;
  if (g > 65536) g = 65536;
  if (g < 1) g = 1;
  return (int)g;
}

void fill_u32(uint32_t* p, uint32_t v, int64_t n, hipStream_t s) {
  if (n > 0) k_fill_u32<<<grid_for(n), 256, 0, s>>>(p, v, n);
}
void fill_f32(float* p, float v, int64_t n, hipStream_t s) {
  if (n > 0) k_fill_f32<<<grid_for(n), 256, 0, s>>>(p, v, n);
}

template <typename T>
__global__ void k_from_f32(const float* src, T* dst, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    St<T>::st(dst, i, src[i]);
}
template <typename T>
__global__ void k_to_f32(const T* src, float* dst, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = St<T>::ld(src, i);
}
template <typename T>
void convert_from_f32(const float* src, T* dst, int64_t n, hipStream_t s) {
  if (n > 0) k_from_f32<T><<<grid_for(n), 256, 0, s>>>(src, dst, n);
}
template <typename T>
void convert_to_f32(const T* src, float* dst, int64_t n, hipStream_t s) {
  if (n > 0) k_to_f32<T><<<grid_for(n), 256, 0, s>>>(src, dst, n);
}
template void convert_from_f32<float>(const float*, float*, int64_t, hipStream_t);
template void convert_from_f32<bf16_t>(const float*, bf16_t*, int64_t, hipStream_t);
template void convert_to_f32<float>(const float*, float*, int64_t, hipStream_t);
template void convert_to_f32<bf16_t>(const bf16_t*, float*, int64_t, hipStream_t);

template <typename T>
__global__ void k_pack_conv(const float* src, T* dst, int d, int C) {
  int64_t n = (int64_t)d * C * 3;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    int64_t o = i / (3 * C);
    int r = (int)(i - o * 3 * C);
    int j = r / C, c = r - j * C;                    // dst[o][j][c]
    St<T>::st(dst, i, src[(o * C + c) * 3 + j]);     // src[o][c][j]
  }
}
template <typename T>
void pack_conv(const float* src, T* dst, int d, int C, hipStream_t s) {
  k_pack_conv<T><<<grid_for((int64_t)d * C * 3), 256, 0, s>>>(src, dst, d, C);
}
template void pack_conv<float>(const float*, float*, int, int, hipStream_t);
template void pack_conv<bf16_t>(const float*, bf16_t*, int, int, hipStream_t);

template <typename T>
__global__ void k_copy_rows(const float* src, int64_t src_ld, T* dst, int64_t dst_ld, int rows,
                            int cols) {
  int64_t n = (int64_t)rows * cols;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    int64_t r = i / cols;
    int c = (int)(i - r * cols);
    St<T>::st(dst, r * dst_ld + c, src[r * src_ld + c]);
  }
}
template <typename T>
void copy_rows_from_f32(const float* src, int64_t src_ld, T* dst, int64_t dst_ld, int rows,
                        int cols, hipStream_t s) {
  if ((int64_t)rows * cols > 0)
    k_copy_rows<T><<<grid_for((int64_t)rows * cols), 256, 0, s>>>(src, src_ld, dst, dst_ld,
                                                                   rows, cols);
}
template void copy_rows_from_f32<float>(const float*, int64_t, float*, int64_t, int, int,
                                        hipStream_t);
template void copy_rows_from_f32<bf16_t>(const float*, int64_t, bf16_t*, int64_t, int, int,
                                         hipStream_t);

// ---------------------------------------------------------------------------
// LayerNorm: one wave per row, biased variance, eps 1e-5.  With RES the
// residual branch y is first added into the stream (x += y, written back).
// Rows of d = 256 * Q floats move as float4 (Q per lane).
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ void st4(T* p, float4 v);
template <>
__device__ __forceinline__ void st4<float>(float* p, float4 v) {
  *(float4*)p = v;
}
template <>
__device__ __forceinline__ void st4<bf16_t>(bf16_t* p, float4 v) {
  uint2 u;
  u.x = pack2_bf16(v.x, v.y);
  u.y = pack2_bf16(v.z, v.w);
  *(uint2*)p = u;
}

template <typename T>
__device__ __forceinline__ float4 ld4(const T* p);
template <>
__device__ __forceinline__ float4 ld4<float>(const float* p) {
  return *(const float4*)p;
}
template <>
__device__ __forceinline__ float4 ld4<bf16_t>(const bf16_t* p) {
  const uint2 u = *(const uint2*)p;
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
}

// Residual modes of the LayerNorm kernels: LN_PLAIN normalises x;
// LN_RES adds one branch (x += y1, stored) first; LN_RES_TEMP normalises
// x + y1 without storing the sum; LN_RES2 adds two branches in order
// (x = (x + y1) + y2, stored).  Branch rows are ldy elements apart.
enum LnMode : int { LN_PLAIN = 0, LN_RES = 1, LN_RES_TEMP = 2, LN_RES2 = 3 };

// All of a row's loads (x, branches, gain, bias) are issued before the first
// store, and the reductions stay in VALU lanes (DPP and lane swaps): the
// row's two passes over HBM then overlap instead of alternating with waits.
template <typename T, int Q, int MODE>
__global__ __launch_bounds__(256) void k_layer_norm(float* __restrict__ x,
                                                    const T* __restrict__ y1,
                                                    const T* __restrict__ y2, int64_t ldy,
                                                    int rows, const float* __restrict__ g,
                                                    const float* __restrict__ b,
                                                    T* __restrict__ out) {
  constexpr int d = Q * 256;
  int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  int lane = threadIdx.x & 63;
  if (row >= rows) return;
  float* xr = x + (int64_t)row * d;
  float4 v[Q], t[Q], t2[Q], gg[Q], bb[Q];
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    const int e = (lane + 64 * i) * 4;
    v[i] = *(const float4*)(xr + e);
    if constexpr (MODE != LN_PLAIN) t[i] = ld4<T>(y1 + (int64_t)row * ldy + e);
    if constexpr (MODE == LN_RES2) t2[i] = ld4<T>(y2 + (int64_t)row * ldy + e);
  }
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    const int e = (lane + 64 * i) * 4;
    gg[i] = *(const float4*)(g + e);
    bb[i] = *(const float4*)(b + e);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    if constexpr (MODE != LN_PLAIN)
      v[i] = make_float4(v[i].x + t[i].x, v[i].y + t[i].y, v[i].z + t[i].z, v[i].w + t[i].w);
    if constexpr (MODE == LN_RES2)
      v[i] = make_float4(v[i].x + t2[i].x, v[i].y + t2[i].y, v[i].z + t2[i].z, v[i].w + t2[i].w);
    if constexpr (MODE == LN_RES || MODE == LN_RES2) *(float4*)(xr + (lane + 64 * i) * 4) = v[i];
    s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
  }
  float mean = wave_sum_lanes(s) * (1.0f / d);
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    v[i] = make_float4(v[i].x - mean, v[i].y - mean, v[i].z - mean, v[i].w - mean);
    q += (v[i].x * v[i].x + v[i].y * v[i].y) + (v[i].z * v[i].z + v[i].w * v[i].w);
  }
  float rstd = rsqrtf(wave_sum_lanes(q) * (1.0f / d) + 1e-5f);
  T* o = out + (int64_t)row * d;
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    const int e = (lane + 64 * i) * 4;
    st4<T>(o + e, make_float4(v[i].x * rstd * gg[i].x + bb[i].x, v[i].y * rstd * gg[i].y + bb[i].y,
                              v[i].z * rstd * gg[i].z + bb[i].z, v[i].w * rstd * gg[i].w + bb[i].w));
  }
}

// Any d that is a multiple of 64: two passes over global memory (the sum
// is formed in the same order as above; LN_RES_TEMP recomputes it).
template <typename T, int MODE>
__global__ __launch_bounds__(256) void k_layer_norm_any(float* x, const T* y1, const T* y2,
                                                        int64_t ldy, int rows, int d,
                                                        const float* g, const float* b, T* out) {
  int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  int lane = threadIdx.x & 63;
  if (row >= rows) return;
  float* xr = x + (int64_t)row * d;
  auto val = [&](int e) {
    float v = xr[e];
    if constexpr (MODE != LN_PLAIN) v += St<T>::ld(y1, (int64_t)row * ldy + e);
    if constexpr (MODE == LN_RES2) v += St<T>::ld(y2, (int64_t)row * ldy + e);
    return v;
  };
  float s = 0.f;
  for (int e = lane; e < d; e += 64) {
    const float v = val(e);
    if constexpr (MODE == LN_RES || MODE == LN_RES2) xr[e] = v;
    s += v;
  }
  float mean = wave_sum(s) / d;
  auto cur = [&](int e) {
    if constexpr (MODE == LN_RES_TEMP) return val(e);
    else return xr[e];
  };
  float q = 0.f;
  for (int e = lane; e < d; e += 64) {
    float t = cur(e) - mean;
    q += t * t;
  }
  float rstd = rsqrtf(wave_sum(q) / d + 1e-5f);
  T* o = out + (int64_t)row * d;
  for (int e = lane; e < d; e += 64) St<T>::st(o, e, (cur(e) - mean) * rstd * g[e] + b[e]);
}

template <typename T, int MODE>
static void layer_norm_launch(float* x, const T* y1, const T* y2, int64_t ldy, int rows, int d,
                              const float* g, const float* b, T* out, hipStream_t s) {
  if (rows <= 0) return;
  dim3 grid((rows + 3) / 4);
  switch (d) {
    case 512: k_layer_norm<T, 2, MODE><<<grid, 256, 0, s>>>(x, y1, y2, ldy, rows, g, b, out); break;
    case 768: k_layer_norm<T, 3, MODE><<<grid, 256, 0, s>>>(x, y1, y2, ldy, rows, g, b, out); break;
    case 1024: k_layer_norm<T, 4, MODE><<<grid, 256, 0, s>>>(x, y1, y2, ldy, rows, g, b, out); break;
    case 1280: k_layer_norm<T, 5, MODE><<<grid, 256, 0, s>>>(x, y1, y2, ldy, rows, g, b, out); break;
    default: k_layer_norm_any<T, MODE><<<grid, 256, 0, s>>>(x, y1, y2, ldy, rows, d, g, b, out); break;
  }
}

template <typename T>
void layer_norm(const float* x, int rows, int d, const float* g, const float* b, T* out,
                hipStream_t s) {
  layer_norm_launch<T, LN_PLAIN>(const_cast<float*>(x), nullptr, nullptr, 0, rows, d, g, b, out,
                                 s);
}

template <typename T>
void residual_layer_norm(float* x, const T* y1, const T* y2, int64_t ldy, bool store, int rows,
                         int d, const float* g, const float* b, T* out, hipStream_t s) {
  if (y2)
    layer_norm_launch<T, LN_RES2>(x, y1, y2, ldy, rows, d, g, b, out, s);
  else if (store)
    layer_norm_launch<T, LN_RES>(x, y1, nullptr, ldy, rows, d, g, b, out, s);
  else
    layer_norm_launch<T, LN_RES_TEMP>(x, y1, nullptr, ldy, rows, d, g, b, out, s);
}
template void residual_layer_norm<float>(float*, const float*, const float*, int64_t, bool, int,
                                         int, const float*, const float*, float*, hipStream_t);
template void residual_layer_norm<bf16_t>(float*, const bf16_t*, const bf16_t*, int64_t, bool,
                                          int, int, const float*, const float*, bf16_t*,
                                          hipStream_t);
template void layer_norm<float>(const float*, int, int, const float*, const float*, float*,
                                hipStream_t);
template void layer_norm<bf16_t>(const float*, int, int, const float*, const float*, bf16_t*,
                                 hipStream_t);

// ---------------------------------------------------------------------------
// Decoder input: token embedding + learned position embedding.
// ---------------------------------------------------------------------------
template <typename T>
__global__ void k_embed(const T* tok_emb, const float* pos_emb, const int32_t* tokens,
                        const int32_t* pos, int d, float* h) {
  int b = blockIdx.x;
  int64_t t = tokens[b], p = pos[b];
  for (int j = threadIdx.x; j < d; j += blockDim.x)
    h[(int64_t)b * d + j] = St<T>::ld(tok_emb, t * d + j) + pos_emb[p * d + j];
}
template <typename T>
void embed(const T* tok_emb, const float* pos_emb, const int32_t* tokens, const int32_t* pos,
           int D, int d, float* h, hipStream_t s) {
  if (D > 0) k_embed<T><<<D, 256, 0, s>>>(tok_emb, pos_emb, tokens, pos, d, h);
}
template void embed<float>(const float*, const float*, const int32_t*, const int32_t*, int, int,
                           float*, hipStream_t);
template void embed<bf16_t>(const bf16_t*, const float*, const int32_t*, const int32_t*, int,
                            int, float*, hipStream_t);

// ---------------------------------------------------------------------------
// Log-mel front-end.
//
// One block handles MEL_FR consecutive frames of one clip.  The block stages
// the samples its frames cover (reflect padding at both ends of the 30-s
// segment, zeros past the clip's own samples) in LDS and computes each
// frame's 400-point DFT of the windowed samples as a mixed-radix FFT,
// 400 = 16 x 25 (Cooley-Tukey with n = 25 n1 + n2, k = k1 + 16 k2):
//   1. for every n2, the 16-point DFT over n1 of the real sequence
//      y[25 n1 + n2], bins k1 = 0 .. 8 (folding y[n1] +- y[16 - n1]), times
//      the twiddle e^{-2 pi i k1 n2 / 400};
//   2. for k1 = 0 .. 8, the 25-point DFT over n2, itself 5 x 5 (two passes of
//      5-point butterflies with the e^{-2 pi i j1 m2 / 25} twiddles between).
// The input is real, so X[400 - k] = conj X[k]: bin (16 - k1) + 16 k2 is
// the conjugate of bin k1 + 16 (24 - k2), and columns k1 = 0 .. 8 give every
// bin's power -- column k1 writes bin k when k <= 200, else bin 400 - k
// (columns 0 and 8 are their own mirror images and write k <= 200 only).
// The block then applies the mel filters (each filter's nonzero bin range
// only), takes log10 with the 1e-10 floor, and stores the group's maximum
// (a plain store per group: the normalisation reduces a clip's groups, so
// there is no atomic for the blocks working on one clip to queue on).
// ---------------------------------------------------------------------------
constexpr int MEL_FR = kMelGroupFrames;
constexpr int MEL_SEG = (MEL_FR - 1) * kHop + kNFFT;   // 2800 samples
constexpr int MEL_COLS = 9;                            // stage-1 bins k1 = 0 .. 8
// float2 stride of one frame's stage-1 output [25][MEL_COLS], padded to 9
// mod 32 so that stage 2's lanes (frame, k1) = (t / 9, t % 9) read 32
// consecutive words per half-wave
constexpr int MEL_FST = 25 * MEL_COLS + 8;

// Where a clip's samples are: device arrays of pointers and lengths, or the
// same lists carried in the kernel arguments (MelClipArgs).
struct ClipsInMemory {
  const float* const* ptrs;
  const int64_t* n;
  __device__ const float* ptr(int i) const { return ptrs[i]; }
  __device__ int64_t len(int i) const { return n[i]; }
};
struct ClipsInArgs {
  MelClipArgs a;
  __device__ const float* ptr(int i) const { return a.ptr[i]; }
  __device__ int64_t len(int i) const { return a.n[i]; }
};

// cos / sin of 2 pi j / 16 and 2 pi t / 25 (the inner radices' twiddles, as
// literal constants so the unrolled butterflies need no table reads)
__device__ constexpr float kC16[16] = {1.0f, 0.92387953251128674f, 0.70710678118654757f, 0.38268343236508984f, 0.0f, -0.38268343236508973f, -0.70710678118654746f, -0.92387953251128674f, -1.0f, -0.92387953251128685f, -0.70710678118654768f, -0.38268343236509034f, 0.0f, 0.38268343236509000f, 0.70710678118654735f, 0.92387953251128652f};
__device__ constexpr float kS16[16] = {0.0f, 0.38268343236508978f, 0.70710678118654746f, 0.92387953251128674f, 1.0f, 0.92387953251128674f, 0.70710678118654757f, 0.38268343236508989f, 0.0f, -0.38268343236508967f, -0.70710678118654746f, -0.92387953251128652f, -1.0f, -0.92387953251128663f, -0.70710678118654768f, -0.38268343236509039f};
__device__ constexpr float kC25[25] = {1.0f, 0.96858316112863108f, 0.87630668004386358f, 0.72896862742141155f, 0.53582679497899655f, 0.30901699437494745f, 0.06279051952931353f, -0.18738131458572460f, -0.42577929156507272f, -0.63742398974868975f, -0.80901699437494734f, -0.92977648588825135f, -0.99211470131447776f, -0.99211470131447788f, -0.92977648588825146f, -0.80901699437494778f, -0.63742398974868952f, -0.42577929156507216f, -0.18738131458572463f, 0.06279051952931283f, 0.30901699437494723f, 0.53582679497899677f, 0.72896862742141122f, 0.87630668004386314f, 0.96858316112863097f};
__device__ constexpr float kS25[25] = {0.0f, 0.24868988716485479f, 0.48175367410171532f, 0.68454710592868862f, 0.84432792550201508f, 0.95105651629515353f, 0.99802672842827156f, 0.98228725072868872f, 0.90482705246601947f, 0.77051324277578925f, 0.58778525229247325f, 0.36812455268467814f, 0.12533323356430454f, -0.12533323356430429f, -0.36812455268467792f, -0.58778525229247269f, -0.77051324277578936f, -0.90482705246601980f, -0.98228725072868872f, -0.99802672842827156f, -0.95105651629515364f, -0.84432792550201496f, -0.68454710592868895f, -0.48175367410171610f, -0.24868988716485535f};

// 5-point DFT A_j = sum_m a_m e^{-2 pi i j m / 5} of (re, im) pairs in place.
__device__ __forceinline__ void dft5(float* ar, float* ai) {
  const float c1 = 0.30901699437494742f, c2 = -0.80901699437494742f;   // cos(2pi/5), cos(4pi/5)
  const float s1 = 0.95105651629515357f, s2 = 0.58778525229247313f;    // sin(2pi/5), sin(4pi/5)
  const float t1r = ar[1] + ar[4], t1i = ai[1] + ai[4], t3r = ar[1] - ar[4], t3i = ai[1] - ai[4];
  const float t2r = ar[2] + ar[3], t2i = ai[2] + ai[3], t4r = ar[2] - ar[3], t4i = ai[2] - ai[3];
  const float b1r = ar[0] + c1 * t1r + c2 * t2r, b1i = ai[0] + c1 * t1i + c2 * t2i;
  const float b2r = ar[0] + c2 * t1r + c1 * t2r, b2i = ai[0] + c2 * t1i + c1 * t2i;
  const float d1r = s1 * t3r + s2 * t4r, d1i = s1 * t3i + s2 * t4i;
  const float d2r = s2 * t3r - s1 * t4r, d2i = s2 * t3i - s1 * t4i;
  ar[0] = ar[0] + t1r + t2r;
  ai[0] = ai[0] + t1i + t2i;
  ar[1] = b1r + d1i; ai[1] = b1i - d1r;     // b1 - i d1
  ar[4] = b1r - d1i; ai[4] = b1i + d1r;     // b1 + i d1
  ar[2] = b2r + d2i; ai[2] = b2i - d2r;     // b2 - i d2
  ar[3] = b2r - d2i; ai[3] = b2i + d2r;     // b2 + i d2
}

// A group is MEL_FR consecutive frames of one clip; the grid walks the
// groups persistently (group g, g + gridDim.x, ...), and while one group is
// transformed the samples of the block's next group are already loading into
// registers (MEL_PT per thread), so the global latency hides behind the FFT.
constexpr int MEL_GROUPS = kMelGroups;                         // groups per clip
// clips per launch: their pointers and lengths sit in LDS, read there by
// every group (LDS waits are independent of the loads and stores in flight)
constexpr int MEL_LAUNCH_CLIPS = 256;
constexpr int MEL_PT = (MEL_SEG + 255) / 256;                // samples per thread

template <class Clips>
__global__ __launch_bounds__(256) void k_log_mel(Clips clips, int n_clips, int n_mels,
                                                 MelTables tb, float* mel_raw,
                                                 float* group_max) {
  // segment samples and the power spectrum [MEL_FR][kBins + 3] (32 floats
  // of slack: a filter's aligned bin window may run past the last row's
  // bin 200, by at most 19 bins)
  constexpr int SEG_SLOTS = MEL_PT * 256;
  __shared__ float seg[SEG_SLOTS];
  __shared__ __attribute__((aligned(16))) float pwbuf[MEL_FR * (kBins + 3) + 32];
  __shared__ float2 bst[MEL_FR * MEL_FST];               // stage-1 output [f][n2][k1]
  __shared__ float fbw[2 * kBins];                       // packed filter weights (bins past 16)
  __shared__ float red[4];
  __shared__ const float* c_ptr[MEL_LAUNCH_CLIPS];
  __shared__ int32_t c_len[MEL_LAUNCH_CLIPS];             // samples used: at most 30 s
  float (*pw)[kBins + 3] = (float (*)[kBins + 3])pwbuf;
  const int tid = threadIdx.x;
  const int n_items = n_clips * MEL_GROUPS;

  // the power spectrum's padding (bins 201 .. 203 of every row and the
  // slack after the last) is never written by stage 2 and stays zero, so
  // a filter's reads past its own bins multiply a finite value (or zero) by
  // its zero weights, as the dense filterbank product would
  for (int i = tid; i < MEL_FR * (kBins + 3) + 32; i += 256) pwbuf[i] = 0.0f;
  for (int i = tid; i < n_clips; i += 256) {
    const int64_t n = clips.len(i);
    c_ptr[i] = n > 0 ? clips.ptr(i) : tb.window;   // a clip without samples reads the window
    c_len[i] = (int32_t)(n < kSamples30s ? n : kSamples30s);
  }
  // Every table a thread uses depends only on its fixed role, so it sits in
  // registers for the whole kernel instead of being re-read from LDS.
  // Stage-1 role: n2 = tid % 25 for frames tid / 25 and tid / 25 + 10
  // (threads 250 .. 255 idle); the window samples w[25 n1 + n2] and the
  // twiddles e^{-2 pi i k1 n2 / 400} of bins k1 = 1 .. 8.
  const int s1_n2 = tid % 25, s1_fs = tid / 25;
  const bool s1_on = tid < 250;
  float s1_win[16], tw_c[MEL_COLS], tw_s[MEL_COLS];
#pragma unroll
  for (int n1 = 0; n1 < 16; ++n1) s1_win[n1] = tb.window[25 * n1 + s1_n2];
#pragma unroll
  for (int k1 = 1; k1 < MEL_COLS; ++k1) {
    tw_c[k1] = tb.cos_t[k1 * s1_n2];   // k1 n2 < 400
    tw_s[k1] = tb.sin_t[k1 * s1_n2];
  }
  // Mel role: filter m = tid % n_mels for frames tid / n_mels + j * mel_fs
  // (threads past mel_fs * n_mels idle), with the filter's first 16 weights
  // (zero past its end); filters past 16 bins (below 64 mels) take the rest
  // from LDS.  The power rows are read in aligned float4s from the bin
  // m_k0 - m_sh (the multiple of 4 at or below the filter's first bin), so
  // the weight registers start m_sh zeros early: the extra bins add
  // fma(0, p, acc) = acc, the products and their order are unchanged.
  const int mel_fs = 256 / n_mels;   // >= 2
  const int mm = tid % n_mels, m_f = tid / n_mels;
  const bool m_on = tid < mel_fs * n_mels;
  const int m_k0 = tb.fb_range[3 * mm], m_cnt = m_on ? tb.fb_range[3 * mm + 1] : 0;
  const int m_off = tb.fb_range[3 * mm + 2];
  const int m_sh = m_k0 & 3;
  float m_w[20];
#pragma unroll
  for (int i = 0; i < 20; ++i) {
    const int j = i - m_sh;
    m_w[i] = j >= 0 && j < m_cnt && j < 16 ? tb.fb[m_off + j] : 0.0f;
  }
  // float4 reads a frame needs: the wave's widest aligned window
  int wave_cnt = m_on ? (m_sh + min(m_cnt, 16) + 3) / 4 : 0;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) wave_cnt = max(wave_cnt, __shfl_xor(wave_cnt, o, 64));
  wave_cnt = __builtin_amdgcn_readfirstlane(wave_cnt);
  {
    const int nw = tb.fb_range[3 * (n_mels - 1) + 2] + tb.fb_range[3 * (n_mels - 1) + 1];
    for (int i = tid; i < nw; i += 256) fbw[i] = tb.fb[i];   // <= 2 x 201
  }
  // Land the table loads here, once: their first uses sit in branches
  // inside the group loop, where the compiler's wait analysis cannot see
  // that they completed and would otherwise wait for every load and store
  // in flight at each of them.
#pragma unroll
  for (int i = 0; i < 16; ++i) asm volatile("" : "+v"(s1_win[i]));
#pragma unroll
  for (int i = 0; i < 20; ++i) asm volatile("" : "+v"(m_w[i]));
#pragma unroll
  for (int i = 1; i < MEL_COLS; ++i) asm volatile("" : "+v"(tw_c[i]), "+v"(tw_s[i]));

  // Group `it`'s segment starts at sample f0 * kHop - kNFFT / 2 of its clip;
  // it is interior when it needs neither reflection nor zeros (all of it
  // inside the clip's own samples), the common case, which takes plain
  // loads at constant offsets.  Slot u of thread tid is segment sample
  // tid + 256 u; slots past MEL_SEG (the last 16 of 256 MEL_PT) are valid
  // samples too and land in LDS beyond the segment, unread.
  auto seg_start = [&](int f0) { return f0 * kHop - kNFFT / 2; };
  auto interior = [&](int start, int n) { return start >= 0 && start + MEL_PT * 256 <= n; };
  // sample index of slot u at a segment edge (reflect padding at both ends
  // of the 30-s segment)
  auto edge_index = [&](int start, int u) {
    int sidx = start + tid + u * 256;
    if (sidx < 0) sidx = -sidx;
    if (sidx >= kSamples30s) sidx = 2 * (kSamples30s - 1) - sidx;
    return sidx;
  };
  // samples of group `it` into registers.  Every load is unconditional (at
  // an edge the index is clamped into the clip's samples; the zeros past
  // them are a select at use), so all MEL_PT loads are in flight at once
  // rather than each waited on in its own branch.
  auto fetch = [&](int it, float (&r)[MEL_PT]) {
    const int clip = it / MEL_GROUPS, f0 = (it - clip * MEL_GROUPS) * MEL_FR;
    const int n = c_len[clip];
    typedef const __attribute__((address_space(1))) float* gptr;   // global memory
    const gptr x = (gptr)c_ptr[clip];
    const int start = seg_start(f0);
    if (interior(start, n)) {
#pragma unroll
      for (int u = 0; u < MEL_PT; ++u) r[u] = x[start + tid + u * 256];
    } else {
      const int last = n > 0 ? n - 1 : 0;
#pragma unroll
      for (int u = 0; u < MEL_PT; ++u) r[u] = x[min(edge_index(start, u), last)];
    }
  };
  // stage 1 for frame f of the group: the 16-point DFT over n1 of the
  // windowed y[25 n1 + n2], twiddled, into row (f, n2) of the stage-1 output
  auto stage1 = [&](int f) {
    float y[16];
#pragma unroll
    for (int n1 = 0; n1 < 16; ++n1) y[n1] = s1_win[n1] * seg[f * kHop + 25 * n1 + s1_n2];
    float sp[8], dm[8];                       // y[m] + y[16 - m], y[m] - y[16 - m] (m = 1 .. 7)
#pragma unroll
    for (int m = 1; m < 8; ++m) {
      sp[m] = y[m] + y[16 - m];
      dm[m] = y[m] - y[16 - m];
    }
    float2* row = bst + f * MEL_FST + s1_n2 * MEL_COLS;
#pragma unroll
    for (int k1 = 0; k1 < MEL_COLS; ++k1) {
      float re = y[0] + ((k1 & 1) ? -y[8] : y[8]), im = 0.f;
#pragma unroll
      for (int m = 1; m < 8; ++m) {
        const int j = (k1 * m) & 15;          // angle 2 pi j / 16
        re = fmaf(sp[m], kC16[j], re);
        im = fmaf(-dm[m], kS16[j], im);
      }
      // twiddle e^{-2 pi i k1 n2 / 400}
      row[k1] = k1 == 0 ? make_float2(re, im)
                        : make_float2(re * tw_c[k1] + im * tw_s[k1], im * tw_c[k1] - re * tw_s[k1]);
    }
  };
  // the samples of a group from registers into LDS (zeros past the clip's
  // own samples)
  auto put = [&](int it, const float (&r)[MEL_PT]) {
    const int clip = it / MEL_GROUPS, f0 = (it - clip * MEL_GROUPS) * MEL_FR;
    const int n = c_len[clip];
    const int start = seg_start(f0);
    if (interior(start, n)) {
#pragma unroll
      for (int u = 0; u < MEL_PT; ++u) seg[tid + u * 256] = r[u];
    } else {
#pragma unroll
      for (int u = 0; u < MEL_PT; ++u) seg[tid + u * 256] = edge_index(start, u) < n ? r[u] : 0.0f;
    }
  };
  // One group, its samples already in LDS.  The next group's samples load
  // into registers at the start and go to LDS after stage 2 (the segment is
  // free once stage 1 is done), so their latency hides behind two stages
  // and the wait for them comes before this group's stores are issued.
  // Three barriers: stage-1 output ready (segment free), power spectrum and
  // next segment ready, wave maxima ready.
  float nxt[MEL_PT];
  auto process = [&](int it) {
    const int clip = it / MEL_GROUPS, f0 = (it - clip * MEL_GROUPS) * MEL_FR;
    const int it_next = it + (int)gridDim.x;
    if (it_next < n_items) fetch(it_next, nxt);

    if (s1_on) {
      stage1(s1_fs);
      if (s1_fs + 10 < MEL_FR) stage1(s1_fs + 10);
    }
    __syncthreads();

    // stage 2: (frame f, k1 <= 8) -> 25 bins over n2 = 5 m1 + m2, as 5 x 5
    if (tid < MEL_FR * MEL_COLS) {
      const int f = tid / MEL_COLS, k1 = tid - f * MEL_COLS;
      const float2* col = bst + f * MEL_FST + k1;
      float cr[5][5], ci[5][5];               // [m2][j1]
#pragma unroll
      for (int m2 = 0; m2 < 5; ++m2) {
        float ar[5], ai[5];
#pragma unroll
        for (int m1 = 0; m1 < 5; ++m1) {
          const float2 v = col[(5 * m1 + m2) * MEL_COLS];
          ar[m1] = v.x;
          ai[m1] = v.y;
        }
        dft5(ar, ai);                         // over m1 -> j1
#pragma unroll
        for (int j1 = 0; j1 < 5; ++j1) {
          const int t = (j1 * m2) % 25;       // e^{-2 pi i j1 m2 / 25}
          const float c = kC25[t], sn = kS25[t];
          cr[m2][j1] = ar[j1] * c + ai[j1] * sn;
          ci[m2][j1] = ai[j1] * c - ar[j1] * sn;
        }
      }
      const bool mirror = k1 >= 1 && k1 <= 7;
#pragma unroll
      for (int j1 = 0; j1 < 5; ++j1) {
        float ar[5], ai[5];
#pragma unroll
        for (int m2 = 0; m2 < 5; ++m2) {
          ar[m2] = cr[m2][j1];
          ai[m2] = ci[m2][j1];
        }
        dft5(ar, ai);                         // over m2 -> j2; k2 = j1 + 5 j2
#pragma unroll
        for (int j2 = 0; j2 < 5; ++j2) {
          const int k = k1 + 16 * (j1 + 5 * j2);
          const float p = ar[j2] * ar[j2] + ai[j2] * ai[j2];
          if (k < kBins) pw[f][k] = p;
          else if (mirror) pw[f][kNFFT - k] = p;
        }
      }
    }
    if (it_next < n_items) put(it_next, nxt);
    __syncthreads();

    // filterbank, log10 with the 1e-10 floor, the group's maximum; each
    // frame reads NB4 aligned float4s of bins from the filter's aligned
    // start, NB4 the wave's widest window (one straight-line variant per
    // width)
    float local_max = -INFINITY;
    float* const out_g = mel_raw + ((int64_t)clip * kFrames + f0 + m_f) * n_mels + mm;
    auto filters = [&](auto nb) {
      constexpr int NB4 = decltype(nb)::value;
#pragma unroll
      for (int j = 0; j < MEL_FR / 2; ++j) {   // mel_fs >= 2: at most 8 frames per thread
        const int f = m_f + j * mel_fs;
        if (!m_on || f >= MEL_FR || f0 + f >= kFrames) continue;
        const float* prow = pw[f] + m_k0;
        const float4* prow4 = (const float4*)(pw[f] + (m_k0 - m_sh));
        float4 v[NB4];
#pragma unroll
        for (int i = 0; i < NB4; ++i) v[i] = prow4[i];
        // bins outside the lane's own filter carry zero weight
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < NB4; ++i) {
          acc = fmaf(m_w[4 * i], v[i].x, acc);
          acc = fmaf(m_w[4 * i + 1], v[i].y, acc);
          acc = fmaf(m_w[4 * i + 2], v[i].z, acc);
          acc = fmaf(m_w[4 * i + 3], v[i].w, acc);
        }
        for (int i = 16; i < m_cnt; ++i) acc = fmaf(fbw[m_off + i], prow[i], acc);
        // log10 as log2 times log10(2) (the argument is a normal float)
        const float L = __builtin_amdgcn_logf(fmaxf(acc, 1e-10f)) * 0.30102999566398120f;
        out_g[(int64_t)j * mel_fs * n_mels] = L;
        local_max = fmaxf(local_max, L);
      }
    };
    if (wave_cnt <= 1) filters(std::integral_constant<int, 1>());
    else if (wave_cnt <= 2) filters(std::integral_constant<int, 2>());
    else if (wave_cnt <= 3) filters(std::integral_constant<int, 3>());
    else if (wave_cnt <= 4) filters(std::integral_constant<int, 4>());
    else filters(std::integral_constant<int, 5>());
    local_max = wave_max(local_max);
    if ((tid & 63) == 0) red[tid >> 6] = local_max;
    __syncthreads();
    if (tid == 0) group_max[it] = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  };
  __syncthreads();                           // clip lists in LDS
  int it = blockIdx.x;
  if (it < n_items) {
    fetch(it, nxt);
    put(it, nxt);
  }
  __syncthreads();
  for (; it < n_items; it += gridDim.x) process(__builtin_amdgcn_readfirstlane(it));
}

// Resident blocks of the log-mel kernel (two per CU with its LDS).
template <class Clips>
static int mel_grid(int n_clips) {
  static int resident = 0;
  if (!resident) {
    int per_cu = 0, dev = 0, n_cu = 0;
    (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_log_mel<Clips>, 256, 0);
    (void)hipGetDevice(&dev);
    (void)hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
    resident = std::max(1, per_cu) * std::max(1, n_cu);
  }
  return std::min(n_clips * MEL_GROUPS, resident);
}

void log_mel(const float* const* pcm_ptrs, const int64_t* n_samples, int n_clips, int n_mels,
             const MelTables& t, float* mel_raw, float* group_max, hipStream_t s) {
  if (n_clips <= 0 || n_mels <= 0 || n_mels > 128) return;   // the kernel's LDS holds 128 filters
  for (int c0 = 0; c0 < n_clips; c0 += MEL_LAUNCH_CLIPS) {
    const int nc = std::min(MEL_LAUNCH_CLIPS, n_clips - c0);
    k_log_mel<ClipsInMemory><<<mel_grid<ClipsInMemory>(nc), 256, 0, s>>>(
        ClipsInMemory{pcm_ptrs + c0, n_samples + c0}, nc, n_mels, t,
        mel_raw + (size_t)c0 * kFrames * n_mels, group_max + (size_t)c0 * MEL_GROUPS);
  }
}

void log_mel_args(const MelClipArgs& clips, int n_clips, int n_mels, const MelTables& t,
                  float* mel_raw, float* group_max, hipStream_t s) {
  static_assert(kMelArgClips <= MEL_LAUNCH_CLIPS, "one launch");
  if (n_clips <= 0 || n_clips > kMelArgClips || n_mels <= 0 || n_mels > 128) return;
  k_log_mel<ClipsInArgs><<<mel_grid<ClipsInArgs>(n_clips), 256, 0, s>>>(
      ClipsInArgs{clips}, n_clips, n_mels, t, mel_raw, group_max);
}

// Dynamic-range clamp 8 below the clip's maximum, then (x + 4) / 4.  With
// pad_rows = 1 the output has a zero row before and after each clip's 3000
// frames, which the first stem convolution reads as its zero padding.  Rows
// are contiguous in both layouts, so output element i of a clip is input
// element i - pad_rows * n_mels (zero outside the frames): V at a time (V =
// 4 when both buffers are aligned for it; n_mels is a multiple of 8).  The
// clip's maximum is the largest of its groups' maxima, reduced by the first
// wave of each block.
template <typename T, int V>
__global__ __launch_bounds__(256) void k_mel_norm(const float* mel_raw, const float* group_max,
                                                  int n_mels, T* out, int pad_rows) {
  __shared__ float s_floor;
  const int clip = blockIdx.y;
  if (threadIdx.x < 64) {
    float mx = -INFINITY;
    for (int g = threadIdx.x; g < kMelGroups; g += 64)
      mx = fmaxf(mx, group_max[(int64_t)clip * kMelGroups + g]);
    mx = wave_max(mx);
    if (threadIdx.x == 0) s_floor = mx - 8.0f;
  }
  __syncthreads();
  const float floor_v = s_floor;
  const int64_t n_in = (int64_t)kFrames * n_mels, shift = (int64_t)pad_rows * n_mels;
  const int64_t n_out = n_in + 2 * shift;
  const float* src = mel_raw + (int64_t)clip * n_in;
  T* dst = out + (int64_t)clip * n_out;
  for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < n_out / V;
       q += (int64_t)gridDim.x * blockDim.x) {
    const int64_t j = V * q - shift;   // input element of output element V q
    if (V == 4) {
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (j >= 0 && j < n_in) {
        v = *(const float4*)(src + j);
        v.x = (fmaxf(v.x, floor_v) + 4.0f) * 0.25f;
        v.y = (fmaxf(v.y, floor_v) + 4.0f) * 0.25f;
        v.z = (fmaxf(v.z, floor_v) + 4.0f) * 0.25f;
        v.w = (fmaxf(v.w, floor_v) + 4.0f) * 0.25f;
      }
      St<T>::st4(dst, V * q, v);
    } else {
      const float v = j >= 0 && j < n_in ? (fmaxf(src[j], floor_v) + 4.0f) * 0.25f : 0.0f;
      St<T>::st(dst, q, v);
    }
  }
}
template <typename T>
void mel_normalize(const float* mel_raw, const float* group_max, int n_clips, int n_mels,
                   T* out, int pad_rows, hipStream_t s) {
  if (n_clips <= 0) return;
  const bool vec = (uintptr_t)mel_raw % 16 == 0 && (uintptr_t)out % (4 * sizeof(T)) == 0;
  const int V = vec ? 4 : 1;
  const int64_t nv = (int64_t)(kFrames + 2 * pad_rows) * n_mels / V;
  // about 16 vectors per thread, so the maximum's reduction is a small part of a block
  dim3 grid((unsigned)((nv + 256 * 16 - 1) / (256 * 16)), n_clips);
  if (vec)
    k_mel_norm<T, 4><<<grid, 256, 0, s>>>(mel_raw, group_max, n_mels, out, pad_rows);
  else
    k_mel_norm<T, 1><<<grid, 256, 0, s>>>(mel_raw, group_max, n_mels, out, pad_rows);
}
template void mel_normalize<float>(const float*, const float*, int, int, float*, int,
                                   hipStream_t);
template void mel_normalize<bf16_t>(const float*, const float*, int, int, bf16_t*, int,
                                    hipStream_t);

}  // namespace asr
