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

// All of a row's loads (x, y, gain, bias) are issued before the first
// store, and the reductions stay in VALU lanes (DPP and lane swaps): the
// row's two passes over HBM then overlap instead of alternating with waits.
template <typename T, int Q, bool RES>
__global__ __launch_bounds__(256) void k_layer_norm(float* __restrict__ x,
                                                    const T* __restrict__ y, int rows,
                                                    const float* __restrict__ g,
                                                    const float* __restrict__ b,
                                                    T* __restrict__ out) {
  constexpr int d = Q * 256;
  int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  int lane = threadIdx.x & 63;
  if (row >= rows) return;
  float* xr = x + (int64_t)row * d;
  float4 v[Q], t[Q], gg[Q], bb[Q];
#pragma unroll
  for (int i = 0; i < Q; ++i) {
    const int e = (lane + 64 * i) * 4;
    v[i] = *(const float4*)(xr + e);
    if constexpr (RES) t[i] = ld4<T>(y + (int64_t)row * d + e);
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
    if constexpr (RES) {
      v[i] = make_float4(v[i].x + t[i].x, v[i].y + t[i].y, v[i].z + t[i].z, v[i].w + t[i].w);
      *(float4*)(xr + (lane + 64 * i) * 4) = v[i];
    }
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

// Any d that is a multiple of 64: two passes over global memory.
template <typename T, bool RES>
__global__ __launch_bounds__(256) void k_layer_norm_any(float* x, const T* y, int rows,
                                                        int d, const float* g, const float* b,
                                                        T* out) {
  int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  int lane = threadIdx.x & 63;
  if (row >= rows) return;
  float* xr = x + (int64_t)row * d;
  float s = 0.f;
  for (int e = lane; e < d; e += 64) {
    if constexpr (RES) xr[e] += St<T>::ld(y, (int64_t)row * d + e);
    s += xr[e];
  }
  float mean = wave_sum(s) / d;
  float q = 0.f;
  for (int e = lane; e < d; e += 64) {
    float t = xr[e] - mean;
    q += t * t;
  }
  float rstd = rsqrtf(wave_sum(q) / d + 1e-5f);
  T* o = out + (int64_t)row * d;
  for (int e = lane; e < d; e += 64) St<T>::st(o, e, (xr[e] - mean) * rstd * g[e] + b[e]);
}

template <typename T, bool RES>
static void layer_norm_launch(float* x, const T* y, int rows, int d, const float* g,
                              const float* b, T* out, hipStream_t s) {
  if (rows <= 0) return;
  dim3 grid((rows + 3) / 4);
  switch (d) {
    case 512: k_layer_norm<T, 2, RES><<<grid, 256, 0, s>>>(x, y, rows, g, b, out); break;
    case 768: k_layer_norm<T, 3, RES><<<grid, 256, 0, s>>>(x, y, rows, g, b, out); break;
    case 1024: k_layer_norm<T, 4, RES><<<grid, 256, 0, s>>>(x, y, rows, g, b, out); break;
    case 1280: k_layer_norm<T, 5, RES><<<grid, 256, 0, s>>>(x, y, rows, g, b, out); break;
    default: k_layer_norm_any<T, RES><<<grid, 256, 0, s>>>(x, y, rows, d, g, b, out); break;
  }
}

template <typename T>
void layer_norm(const float* x, int rows, int d, const float* g, const float* b, T* out,
                hipStream_t s) {
  layer_norm_launch<T, false>(const_cast<float*>(x), nullptr, rows, d, g, b, out, s);
}

template <typename T>
void residual_layer_norm(float* x, const T* y, int rows, int d, const float* g,
                         const float* b, T* out, hipStream_t s) {
  layer_norm_launch<T, true>(x, y, rows, d, g, b, out, s);
}
template void residual_layer_norm<float>(float*, const float*, int, int, const float*,
                                         const float*, float*, hipStream_t);
template void residual_layer_norm<bf16_t>(float*, const bf16_t*, int, int, const float*,
                                          const float*, bf16_t*, hipStream_t);
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
//      y[25 n1 + n2] (bins 0 .. 8 by folding y[n1] +- y[16 - n1]; bins
//      9 .. 15 are the conjugates of bins 7 .. 1), times the twiddle
//      e^{-2 pi i k1 n2 / 400};
//   2. for every k1, the 25-point DFT over n2, itself 5 x 5 (two passes of
//      5-point butterflies with the e^{-2 pi i j1 m2 / 25} twiddles between);
// bins k = k1 + 16 k2 <= 200 give the power spectrum.  The block then
// applies the mel filters (each filter's nonzero bin range only), takes
// log10 with the 1e-10 floor, and folds its maximum into the clip's maximum
// with an atomic max on order-preserving integer keys.
// ---------------------------------------------------------------------------
constexpr int MEL_FR = 16;
constexpr int MEL_SEG = (MEL_FR - 1) * kHop + kNFFT;   // 2800 samples
constexpr int MEL_BLD = 17;                            // padded row (float2) of stage-1 output

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
constexpr int MEL_GROUPS = (kFrames + MEL_FR - 1) / MEL_FR;   // groups per clip
constexpr int MEL_PT = (MEL_SEG + 255) / 256;                // samples per thread

template <class Clips>
__global__ __launch_bounds__(256) void k_log_mel(Clips clips, int n_clips, int n_mels,
                                                 MelTables tb, float* mel_raw,
                                                 uint32_t* clip_max) {
  // the samples are dead once stage 1 has read them: the power spectrum
  // [MEL_FR][kBins + 3] reuses their LDS (16 floats of slack: a filter's
  // 16-bin window may start at bin 200 of the last row)
  constexpr int SEGPW = (MEL_SEG > MEL_FR * (kBins + 3) ? MEL_SEG : MEL_FR * (kBins + 3)) + 16;
  __shared__ float segpw[SEGPW];
  __shared__ float2 bst[MEL_FR * 25 * MEL_BLD];          // stage-1 output [f][n2][k1]
  __shared__ float fbw[2 * kBins];                       // packed filter weights (bins past 16)
  __shared__ float red[4];
  float* seg = segpw;
  float (*pw)[kBins + 3] = (float (*)[kBins + 3])segpw;
  const int tid = threadIdx.x;
  const int n_items = n_clips * MEL_GROUPS;

  // Every table a thread uses depends only on its fixed role, so it sits in
  // registers for the whole kernel instead of being re-read from LDS.
  // Stage-1 role: n2 = tid % 25 for frames tid / 25 and tid / 25 + 10
  // (threads 250 .. 255 idle); the window samples w[25 n1 + n2] and the
  // twiddles e^{-2 pi i k n2 / 400} of bins k1 = 1 .. 8 and 16 - k1.
  const int s1_n2 = tid % 25, s1_fs = tid / 25;
  const bool s1_on = tid < 250;
  float s1_win[16], tw_c[16], tw_s[16];
#pragma unroll
  for (int n1 = 0; n1 < 16; ++n1) s1_win[n1] = tb.window[25 * n1 + s1_n2];
#pragma unroll
  for (int k1 = 1; k1 < 16; ++k1) {
    const int t = k1 * s1_n2 % kNFFT;
    tw_c[k1] = tb.cos_t[t];
    tw_s[k1] = tb.sin_t[t];
  }
  // Mel role: filter m = tid % n_mels for frames tid / n_mels + j * mel_fs
  // (threads past mel_fs * n_mels idle), with the filter's first 16 weights
  // (zero past its end); filters past 16 bins (below 64 mels) take the rest
  // from LDS.
  const int mel_fs = 256 / n_mels;   // >= 2
  const int mm = tid % n_mels, m_f = tid / n_mels;
  const bool m_on = tid < mel_fs * n_mels;
  const int m_k0 = tb.fb_range[3 * mm], m_cnt = m_on ? tb.fb_range[3 * mm + 1] : 0;
  const int m_off = tb.fb_range[3 * mm + 2];
  float m_w[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) m_w[i] = i < m_cnt ? tb.fb[m_off + i] : 0.0f;
  int wave_cnt = m_cnt;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) wave_cnt = max(wave_cnt, __shfl_xor(wave_cnt, o, 64));
  wave_cnt = __builtin_amdgcn_readfirstlane(wave_cnt);
  {
    const int nw = tb.fb_range[3 * (n_mels - 1) + 2] + tb.fb_range[3 * (n_mels - 1) + 1];
    for (int i = tid; i < nw; i += 256) fbw[i] = tb.fb[i];   // <= 2 x 201
  }

  // sample index (reflect padding at both ends of the 30-s segment) of slot
  // u of group `it`'s segment; slots past MEL_SEG (the last 16 of 256 MEL_PT)
  // map to valid samples too and land in LDS beyond the segment, unread
  auto sample_index = [&](int f0, int u) {
    int64_t sidx = (int64_t)f0 * kHop - kNFFT / 2 + tid + u * 256;
    if (sidx < 0) sidx = -sidx;
    if (sidx >= kSamples30s) sidx = 2 * (int64_t)(kSamples30s - 1) - sidx;
    return sidx;
  };
  // samples of group `it` into registers.  Every load is unconditional (the
  // index is clamped into the clip, and a clip without samples reads the
  // window table instead) and the zeros past the clip's own samples are a
  // select at use, so all MEL_PT loads are in flight at once rather than
  // each waited on in its own branch.
  auto fetch = [&](int it, float (&r)[MEL_PT]) {
    const int clip = it / MEL_GROUPS, f0 = (it - clip * MEL_GROUPS) * MEL_FR;
    const int64_t n = clips.len(clip);
    typedef const __attribute__((address_space(1))) float* gptr;   // global memory
    const gptr x = (gptr)(n > 0 ? clips.ptr(clip) : tb.window);
    const int64_t last = n > 0 ? n - 1 : 0;
#pragma unroll
    for (int u = 0; u < MEL_PT; ++u) {
      const int64_t sidx = sample_index(f0, u);
      r[u] = x[sidx < last ? sidx : last];
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
    float2* row = bst + (f * 25 + s1_n2) * MEL_BLD;
#pragma unroll
    for (int k1 = 0; k1 <= 8; ++k1) {
      float re = y[0] + ((k1 & 1) ? -y[8] : y[8]), im = 0.f;
#pragma unroll
      for (int m = 1; m < 8; ++m) {
        const int j = (k1 * m) & 15;          // angle 2 pi j / 16
        re = fmaf(sp[m], kC16[j], re);
        im = fmaf(-dm[m], kS16[j], im);
      }
      if (k1 == 0) {
        row[0] = make_float2(re, im);
      } else {
        // twiddle e^{-2 pi i k1 n2 / 400} on bin k1 and (conjugate input) on bin 16 - k1
        row[k1] = make_float2(re * tw_c[k1] + im * tw_s[k1], im * tw_c[k1] - re * tw_s[k1]);
        if (k1 <= 7) {                        // conj(A) = (re, -im)
          const int k2 = 16 - k1;
          row[k2] = make_float2(re * tw_c[k2] - im * tw_s[k2], -im * tw_c[k2] - re * tw_s[k2]);
        }
      }
    }
  };
  // one group: its samples (in `cur`) into LDS, the next group's samples
  // into `nxt`, then the transform and the filterbank
  auto process = [&](int it, const float (&cur)[MEL_PT], float (&nxt)[MEL_PT]) {
    const int clip = it / MEL_GROUPS, f0 = (it - clip * MEL_GROUPS) * MEL_FR;
    __syncthreads();                         // the previous group is done with the LDS
    static_assert(MEL_PT * 256 <= SEGPW, "segment slots");
    {
      const int64_t n = clips.len(clip);
#pragma unroll
      for (int u = 0; u < MEL_PT; ++u) seg[tid + u * 256] = sample_index(f0, u) < n ? cur[u] : 0.0f;
    }
    if (it + (int)gridDim.x < n_items) fetch(it + gridDim.x, nxt);
    __syncthreads();

    if (s1_on) {
      stage1(s1_fs);
      if (s1_fs + 10 < MEL_FR) stage1(s1_fs + 10);
    }
    __syncthreads();

    // stage 2: (frame f, k1) -> 25 bins over n2 = 5 m1 + m2, as 5 x 5
    {
      const int f = tid >> 4, k1 = tid & 15;
      float cr[5][5], ci[5][5];               // [m2][j1]
#pragma unroll
      for (int m2 = 0; m2 < 5; ++m2) {
        float ar[5], ai[5];
#pragma unroll
        for (int m1 = 0; m1 < 5; ++m1) {
          const float2 v = bst[(f * 25 + 5 * m1 + m2) * MEL_BLD + k1];
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
          if (k < kBins) pw[f][k] = ar[j2] * ar[j2] + ai[j2] * ai[j2];
        }
      }
    }
    __syncthreads();

    // filterbank, log10 with the 1e-10 floor, the group's maximum; each
    // frame reads NB bins from the filter's first, NB the widest filter of
    // the wave rounded up (one straight-line variant per width)
    float local_max = -INFINITY;
    auto filters = [&](auto nb) {
      constexpr int NB = decltype(nb)::value;
#pragma unroll
      for (int j = 0; j < MEL_FR / 2; ++j) {   // mel_fs >= 2: at most 8 frames per thread
        const int f = m_f + j * mel_fs;
        if (!m_on || f >= MEL_FR || f0 + f >= kFrames) continue;
        const float* prow = pw[f] + m_k0;
        float v[NB];
#pragma unroll
        for (int i = 0; i < NB; ++i) v[i] = prow[i];
        // bins past the lane's own filter carry zero weight; the select
        // keeps whatever they hold out of the sum
        float acc = 0.f;
#pragma unroll
        for (int i = 0; i < NB; ++i) acc = fmaf(m_w[i], i < m_cnt ? v[i] : 0.0f, acc);
        for (int i = 16; i < m_cnt; ++i) acc = fmaf(fbw[m_off + i], prow[i], acc);
        const float L = log10f(fmaxf(acc, 1e-10f));
        mel_raw[((int64_t)clip * kFrames + f0 + f) * n_mels + mm] = L;
        local_max = fmaxf(local_max, L);
      }
    };
    if (wave_cnt <= 2) filters(std::integral_constant<int, 2>());
    else if (wave_cnt <= 4) filters(std::integral_constant<int, 4>());
    else if (wave_cnt <= 8) filters(std::integral_constant<int, 8>());
    else if (wave_cnt <= 12) filters(std::integral_constant<int, 12>());
    else filters(std::integral_constant<int, 16>());
    local_max = wave_max(local_max);
    if ((tid & 63) == 0) red[tid >> 6] = local_max;
    __syncthreads();
    if (tid == 0) {
      float mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
      atomicMax(clip_max + clip, ordered_u32(mx));
    }
  };
  // ping-pong between two register sets, so no copy forces the next group's
  // loads to land before this group's work
  float sa[MEL_PT], sb[MEL_PT];
  int it = blockIdx.x;
  if (it < n_items) fetch(it, sa);
  while (it < n_items) {
    process(it, sa, sb);
    it += gridDim.x;
    if (it >= n_items) break;
    process(it, sb, sa);
    it += gridDim.x;
  }
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
             const MelTables& t, float* mel_raw, uint32_t* clip_max, hipStream_t s) {
  if (n_clips <= 0 || n_mels <= 0 || n_mels > 128) return;   // the kernel's LDS holds 128 filters
  fill_u32(clip_max, 0u, n_clips, s);
  k_log_mel<ClipsInMemory><<<mel_grid<ClipsInMemory>(n_clips), 256, 0, s>>>(
      ClipsInMemory{pcm_ptrs, n_samples}, n_clips, n_mels, t, mel_raw, clip_max);
}

void log_mel_args(const MelClipArgs& clips, int n_clips, int n_mels, const MelTables& t,
                  float* mel_raw, uint32_t* clip_max, hipStream_t s) {
  if (n_clips <= 0 || n_mels <= 0 || n_mels > 128) return;
  fill_u32(clip_max, 0u, n_clips, s);
  k_log_mel<ClipsInArgs><<<mel_grid<ClipsInArgs>(n_clips), 256, 0, s>>>(
      ClipsInArgs{clips}, n_clips, n_mels, t, mel_raw, clip_max);
}

// Dynamic-range clamp 8 below the clip's maximum, then (x + 4) / 4.  With
// pad_rows = 1 the output has a zero row before and after each clip's 3000
// frames, which the first stem convolution reads as its zero padding.
template <typename T>
__global__ void k_mel_norm(const float* mel_raw, const uint32_t* clip_max, int n_mels, T* out,
                           int pad_rows) {
  int clip = blockIdx.y;
  int rows_out = kFrames + 2 * pad_rows;
  float floor_v = from_ordered_u32(clip_max[clip]) - 8.0f;
  int64_t n = (int64_t)rows_out * n_mels;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    int64_t r = i / n_mels;
    int m = (int)(i - r * n_mels);
    int64_t frame = r - pad_rows;
    float v = 0.f;
    if (frame >= 0 && frame < kFrames) {
      float L = mel_raw[((int64_t)clip * kFrames + frame) * n_mels + m];
      v = (fmaxf(L, floor_v) + 4.0f) * 0.25f;
    }
    St<T>::st(out, (int64_t)clip * n + i, v);
  }
}
template <typename T>
void mel_normalize(const float* mel_raw, const uint32_t* clip_max, int n_clips, int n_mels,
                   T* out, int pad_rows, hipStream_t s) {
  if (n_clips <= 0) return;
  int64_t n = (int64_t)(kFrames + 2 * pad_rows) * n_mels;
  dim3 grid((unsigned)((n + 255) / 256 > 4096 ? 4096 : (n + 255) / 256), n_clips);
  k_mel_norm<T><<<grid, 256, 0, s>>>(mel_raw, clip_max, n_mels, out, pad_rows);
}
template void mel_normalize<float>(const float*, const uint32_t*, int, int, float*, int,
                                   hipStream_t);
template void mel_normalize<bf16_t>(const float*, const uint32_t*, int, int, bf16_t*, int,
                                    hipStream_t);

}  // namespace asr
