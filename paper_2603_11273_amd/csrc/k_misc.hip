// Elementwise and row kernels: fills, conversions, weight packing, LayerNorm,
// decoder embedding, and the log-mel front-end.
#include "asr_device.h"

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
// segment, zeros past the clip's own samples) in LDS, each of the first 201
// threads computes one DFT bin for all MEL_FR frames from a 400-entry
// cos/sin table (the window is folded into the twiddle), and the block then
// applies the mel filters (each filter's nonzero bin range only), takes
// log10 with the 1e-10 floor, and folds its maximum into the clip's maximum
// with an atomic max on order-preserving integer keys.
// ---------------------------------------------------------------------------
constexpr int MEL_FR = 16;
constexpr int MEL_SEG = (MEL_FR - 1) * kHop + kNFFT;   // 2800 samples

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

template <class Clips>
__global__ __launch_bounds__(256) void k_log_mel(Clips clips, int n_mels, MelTables tb,
                                                 float* mel_raw, uint32_t* clip_max) {
  __shared__ float seg[MEL_SEG];
  __shared__ float wc[kNFFT], ws[kNFFT];
  __shared__ float pw[MEL_FR][kBins + 3];
  __shared__ float red[4];
  const int clip = blockIdx.y;
  const int f0 = blockIdx.x * MEL_FR;
  const float* x = clips.ptr(clip);
  const int64_t n = clips.len(clip);
  const int tid = threadIdx.x;

  for (int i = tid; i < MEL_SEG; i += 256) {
    int64_t sidx = (int64_t)f0 * kHop - kNFFT / 2 + i;
    if (sidx < 0) sidx = -sidx;                                   // reflect at the start
    if (sidx >= kSamples30s) sidx = 2 * (int64_t)(kSamples30s - 1) - sidx;   // and the end
    seg[i] = (sidx < n) ? x[sidx] : 0.0f;
  }
  for (int i = tid; i < kNFFT; i += 256) {
    wc[i] = tb.cos_t[i];
    ws[i] = tb.sin_t[i];
  }
  __syncthreads();

  if (tid < kBins) {
    const int k = tid;
    float re[MEL_FR], im[MEL_FR];
#pragma unroll
    for (int f = 0; f < MEL_FR; ++f) re[f] = im[f] = 0.f;
    int j = 0;                                                    // (k * n) mod 400
    for (int nn = 0; nn < kNFFT; ++nn) {
      float w = tb.window[nn];
      float c = wc[j] * w, sn = ws[j] * w;
#pragma unroll
      for (int f = 0; f < MEL_FR; ++f) {
        float v = seg[f * kHop + nn];
        re[f] = fmaf(v, c, re[f]);
        im[f] = fmaf(v, sn, im[f]);
      }
      j += k;
      if (j >= kNFFT) j -= kNFFT;
    }
#pragma unroll
    for (int f = 0; f < MEL_FR; ++f) pw[f][k] = re[f] * re[f] + im[f] * im[f];
  }
  __syncthreads();

  float local_max = -INFINITY;
  const int total = MEL_FR * n_mels;
  for (int idx = tid; idx < total; idx += 256) {
    int f = idx / n_mels, m = idx - f * n_mels;
    int frame = f0 + f;
    if (frame >= kFrames) continue;
    int k0 = tb.fb_range[2 * m], cnt = tb.fb_range[2 * m + 1];
    const float* wrow = tb.fb + (int64_t)m * kBins;
    float acc = 0.f;
    for (int k = k0; k < k0 + cnt; ++k) acc = fmaf(wrow[k], pw[f][k], acc);
    float L = log10f(fmaxf(acc, 1e-10f));
    mel_raw[((int64_t)clip * kFrames + frame) * n_mels + m] = L;
    local_max = fmaxf(local_max, L);
  }
  local_max = wave_max(local_max);
  if ((tid & 63) == 0) red[tid >> 6] = local_max;
  __syncthreads();
  if (tid == 0) {
    float m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    atomicMax(clip_max + clip, ordered_u32(m));
  }
}

void log_mel(const float* const* pcm_ptrs, const int64_t* n_samples, int n_clips, int n_mels,
             const MelTables& t, float* mel_raw, uint32_t* clip_max, hipStream_t s) {
  if (n_clips <= 0) return;
  fill_u32(clip_max, 0u, n_clips, s);
  dim3 grid((kFrames + MEL_FR - 1) / MEL_FR, n_clips);
  k_log_mel<ClipsInMemory><<<grid, 256, 0, s>>>(ClipsInMemory{pcm_ptrs, n_samples}, n_mels, t,
                                                mel_raw, clip_max);
}

void log_mel_args(const MelClipArgs& clips, int n_clips, int n_mels, const MelTables& t,
                  float* mel_raw, uint32_t* clip_max, hipStream_t s) {
  if (n_clips <= 0) return;
  fill_u32(clip_max, 0u, n_clips, s);
  dim3 grid((kFrames + MEL_FR - 1) / MEL_FR, n_clips);
  k_log_mel<ClipsInArgs><<<grid, 256, 0, s>>>(ClipsInArgs{clips}, n_mels, t, mel_raw, clip_max);
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
