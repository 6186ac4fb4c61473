// Attention kernels.
//
//  * flash_attn_bf16: encoder self-attention over the 1500 positions of a
//    30-s segment (no mask), MFMA-based.  Each wave owns 32 queries; K and
//    V^T tiles of 64 keys are staged in LDS and shared by the block's 4
//    waves.  The kernel computes S^T = K Q^T so that, in the MFMA output
//    layout, each lane holds one query's scores for 16 keys: the row max and
//    sum need a single cross-lane exchange, the probabilities feed the
//    O^T = V^T P^T product directly as its B operand, and the per-query
//    rescale is a per-lane multiply.  Softmax runs in fp32 with exp2.
//  * flash_attn_f32: the same result in plain fp32 (one thread per query).
//  * decode self / cross attention: one block per (row, head), streaming the
//    row's cache once: scores for all keys, exact softmax, then the
//    probability-weighted value sum.  The self variant first stores this
//    step's key and value at the slot's position.
#include "asr_device.h"

namespace asr {

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) {
  bf16x8 r;
  __builtin_memcpy(&r, &u, 16);
  return r;
}
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
}

// ---------------------------------------------------------------------------
// Encoder flash attention (bf16)
// ---------------------------------------------------------------------------
constexpr int FA_KT = 64;          // keys per tile
constexpr int FA_LD = 64 + 8;      // padded LDS row

__global__ __launch_bounds__(256) void k_flash_bf16(const bf16_t* __restrict__ qkv,
                                                    bf16_t* __restrict__ out, int n_head) {
  __shared__ __attribute__((aligned(16))) bf16_t Ks[FA_KT * FA_LD];   // [key][dim]
  __shared__ __attribute__((aligned(16))) bf16_t Vt[64 * FA_LD];      // [dim][key]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = blockIdx.y, b = blockIdx.z;
  const int d = n_head * 64, ld3 = 3 * d;
  const bf16_t* base = qkv + (int64_t)b * kCtx * ld3;
  const int qrow = blockIdx.x * 128 + wave * 32 + (lane & 31);
  const bool qvalid = qrow < kCtx;
  const int half = lane >> 5;
  const uint4 z = {0u, 0u, 0u, 0u};

  bf16x8 qf[4];
  {
    const bf16_t* qp = base + (int64_t)(qvalid ? qrow : 0) * ld3 + h * 64 + half * 8;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      qf[kk] = as_bf16x8(qvalid ? *(const uint4*)(qp + kk * 16) : z);
  }
  f32x16 o0, o1;
#pragma unroll
  for (int r = 0; r < 16; ++r) o0[r] = o1[r] = 0.f;
  float m = -INFINITY, l = 0.f;
  const float sc = 0.125f * 1.4426950408889634f;     // 1/sqrt(64) * log2(e)

  for (int k0 = 0; k0 < kCtx; k0 += FA_KT) {
    for (int c = tid; c < FA_KT * 8; c += 256) {
      int key = c >> 3, dc = (c & 7) * 8;
      int gk = k0 + key;
      uint4 kv = z, vv = z;
      if (gk < kCtx) {
        const bf16_t* rp = base + (int64_t)gk * ld3 + h * 64 + dc;
        kv = *(const uint4*)(rp + d);
        vv = *(const uint4*)(rp + 2 * d);
      }
      *(uint4*)&Ks[key * FA_LD + dc] = kv;
      const bf16_t* ve = (const bf16_t*)&vv;
#pragma unroll
      for (int i = 0; i < 8; ++i) Vt[(dc + i) * FA_LD + key] = ve[i];
    }
    __syncthreads();

    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        bf16x8 kf = *(const bf16x8*)&Ks[(kb * 32 + (lane & 31)) * FA_LD + kk * 16 + half * 8];
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], s[kb], 0, 0, 0);
      }
    }
    // s[kb][r]: key k0 + 32 kb + 8 (r/4) + 4 half + r%4, query qrow
    float tmax = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int key = k0 + kb * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
        float v = key < kCtx ? s[kb][r] * sc : -INFINITY;
        s[kb][r] = v;
        tmax = fmaxf(tmax, v);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float mnew = fmaxf(m, tmax);
    const float alpha = exp2f(m - mnew);
    m = mnew;
    float psum = 0.f;
    bf16x8 pb[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        float p[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          p[i] = exp2f(s[kb][hf * 8 + i] - mnew);
          psum += p[i];
        }
        uint4 u = {pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]), pack_bf16x2(p[4], p[5]),
                   pack_bf16x2(p[6], p[7])};
        pb[kb][hf] = as_bf16x8(u);
      }
    l = l * alpha + psum;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      o0[r] *= alpha;
      o1[r] *= alpha;
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const int kbase = kb * 32 + hf * 16 + half * 4;
        const bf16_t* v0 = &Vt[(lane & 31) * FA_LD + kbase];
        const bf16_t* v1 = &Vt[(32 + (lane & 31)) * FA_LD + kbase];
        uint2 a0 = *(const uint2*)v0, a1 = *(const uint2*)(v0 + 8);
        uint2 c0 = *(const uint2*)v1, c1 = *(const uint2*)(v1 + 8);
        bf16x8 vf0 = as_bf16x8(uint4{a0.x, a0.y, a1.x, a1.y});
        bf16x8 vf1 = as_bf16x8(uint4{c0.x, c0.y, c1.x, c1.y});
        o0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf0, pb[kb][hf], o0, 0, 0, 0);
        o1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf1, pb[kb][hf], o1, 0, 0, 0);
      }
    __syncthreads();
  }
  l += __shfl_xor(l, 32, 64);
  if (!qvalid) return;
  const float inv = 1.0f / l;
  bf16_t* op = out + ((int64_t)b * kCtx + qrow) * d + h * 64;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    int d0 = g * 8 + half * 4;
    uint2 w0 = {pack_bf16x2(o0[g * 4 + 0] * inv, o0[g * 4 + 1] * inv),
                pack_bf16x2(o0[g * 4 + 2] * inv, o0[g * 4 + 3] * inv)};
    uint2 w1 = {pack_bf16x2(o1[g * 4 + 0] * inv, o1[g * 4 + 1] * inv),
                pack_bf16x2(o1[g * 4 + 2] * inv, o1[g * 4 + 3] * inv)};
    *(uint2*)(op + d0) = w0;
    *(uint2*)(op + 32 + d0) = w1;
  }
}

void flash_attn_bf16(const bf16_t* qkv, bf16_t* out, int B, int n_head, hipStream_t s) {
  if (B <= 0) return;
  dim3 grid((kCtx + 127) / 128, n_head, B);
  k_flash_bf16<<<grid, 256, 0, s>>>(qkv, out, n_head);
}

// ---------------------------------------------------------------------------
// Encoder attention, fp32 (one thread per query, 32-key tiles in LDS)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(128) void k_flash_f32(const float* __restrict__ qkv,
                                                   float* __restrict__ out, int n_head) {
  constexpr int KT = 32;
  __shared__ float Ksh[KT][64];
  __shared__ float Vsh[KT][64];
  const int h = blockIdx.y, b = blockIdx.z;
  const int d = n_head * 64, ld3 = 3 * d;
  const float* base = qkv + (int64_t)b * kCtx * ld3;
  const int qrow = blockIdx.x * 128 + threadIdx.x;
  const bool qvalid = qrow < kCtx;
  float q[64], o[64];
  const float* qp = base + (int64_t)(qvalid ? qrow : 0) * ld3 + h * 64;
#pragma unroll
  for (int i = 0; i < 64; ++i) {
    q[i] = qp[i] * 0.125f;
    o[i] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int k0 = 0; k0 < kCtx; k0 += KT) {
    for (int c = threadIdx.x; c < KT * 64; c += 128) {
      int key = c >> 6, j = c & 63;
      int gk = k0 + key;
      Ksh[key][j] = gk < kCtx ? base[(int64_t)gk * ld3 + d + h * 64 + j] : 0.f;
      Vsh[key][j] = gk < kCtx ? base[(int64_t)gk * ld3 + 2 * d + h * 64 + j] : 0.f;
    }
    __syncthreads();
    float s[KT];
    float tmax = -INFINITY;
#pragma unroll
    for (int k = 0; k < KT; ++k) {
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < 64; ++i) acc = fmaf(q[i], Ksh[k][i], acc);
      s[k] = (k0 + k < kCtx) ? acc : -INFINITY;
      tmax = fmaxf(tmax, s[k]);
    }
    float mnew = fmaxf(m, tmax);
    float alpha = expf(m - mnew);
    m = mnew;
    l *= alpha;
#pragma unroll
    for (int i = 0; i < 64; ++i) o[i] *= alpha;
#pragma unroll
    for (int k = 0; k < KT; ++k) {
      float p = expf(s[k] - mnew);
      l += p;
#pragma unroll
      for (int i = 0; i < 64; ++i) o[i] = fmaf(p, Vsh[k][i], o[i]);
    }
    __syncthreads();
  }
  if (!qvalid) return;
  float inv = 1.0f / l;
  float* op = out + ((int64_t)b * kCtx + qrow) * d + h * 64;
#pragma unroll
  for (int i = 0; i < 64; ++i) op[i] = o[i] * inv;
}

void flash_attn_f32(const float* qkv, float* out, int B, int n_head, hipStream_t s) {
  if (B <= 0) return;
  dim3 grid((kCtx + 127) / 128, n_head, B);
  k_flash_f32<<<grid, 128, 0, s>>>(qkv, out, n_head);
}

// ---------------------------------------------------------------------------
// Decode attention
// ---------------------------------------------------------------------------
// Loads 8 consecutive head dims of one key/value row as floats.
__device__ __forceinline__ void load8(const float* p, float* v) {
  float4 a = *(const float4*)p, c = *(const float4*)(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = c.x; v[5] = c.y; v[6] = c.z; v[7] = c.w;
}
__device__ __forceinline__ void load8(const bf16_t* p, float* v) {
  uint4 u = *(const uint4*)p;
  v[0] = __uint_as_float(u.x << 16); v[1] = __uint_as_float(u.x & 0xffff0000u);
  v[2] = __uint_as_float(u.y << 16); v[3] = __uint_as_float(u.y & 0xffff0000u);
  v[4] = __uint_as_float(u.z << 16); v[5] = __uint_as_float(u.z & 0xffff0000u);
  v[6] = __uint_as_float(u.w << 16); v[7] = __uint_as_float(u.w & 0xffff0000u);
}

// Block of 256 threads; lane group of 8 lanes per key (8 dims each), 4 waves
// x 8 keys = 32 keys per pass, 4 passes unrolled per loop iteration.
template <typename T, bool SELF>
__global__ __launch_bounds__(256) void k_decode_attn(const T* __restrict__ src, T* cache,
                                                     int64_t slot_stride, int64_t layer_off,
                                                     const int32_t* slots, const int32_t* pos,
                                                     int n_head, T* __restrict__ out) {
  constexpr int CTX = SELF ? kTextCtx : kCtx;
  __shared__ float qs[64];
  __shared__ float sc[CTX];
  __shared__ float red[4];
  __shared__ float ored[4][64];
  const int h = blockIdx.x, row = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = n_head * 64;
  const int ldsrc = SELF ? 3 * d : d;
  const int slot = slots[row];
  const int n = SELF ? pos[row] + 1 : kCtx;
  T* kb = cache + (int64_t)slot * slot_stride + layer_off + (int64_t)h * CTX * 64;
  T* vb = kb + (int64_t)n_head * CTX * 64;
  const T* srow = src + (int64_t)row * ldsrc + h * 64;

  if (tid < 64) qs[tid] = St<T>::ld(srow, tid) * 0.125f;
  if (SELF && tid < 128) {                      // store this step's k, v at position n-1
    int j = tid & 63;
    if (tid < 64)
      kb[(int64_t)(n - 1) * 64 + j] = srow[d + j];
    else
      vb[(int64_t)(n - 1) * 64 + j] = srow[2 * d + j];
  }
  __syncthreads();

  const int sub = lane >> 3, dc = (lane & 7) * 8;
  float qv[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) qv[i] = qs[dc + i];

  // scores
  for (int g0 = 0; g0 < n; g0 += 128) {
    float part[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      int key = g0 + u * 32 + wave * 8 + sub;
      part[u] = 0.f;
      if (key < n) {
        const T* kp = (SELF && key == n - 1) ? (srow + d) : (kb + (int64_t)key * 64);
        float kv[8];
        load8(kp + dc, kv);
#pragma unroll
        for (int i = 0; i < 8; ++i) part[u] = fmaf(qv[i], kv[i], part[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      float p = part[u];
      p += __shfl_xor(p, 1, 64);
      p += __shfl_xor(p, 2, 64);
      p += __shfl_xor(p, 4, 64);
      int key = g0 + u * 32 + wave * 8 + sub;
      if ((lane & 7) == 0 && key < n) sc[key] = p;
    }
  }
  __syncthreads();

  float mx = -INFINITY;
  for (int k = tid; k < n; k += 256) mx = fmaxf(mx, sc[k]);
  mx = wave_max(mx);
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float sum = 0.f;
  for (int k = tid; k < n; k += 256) {
    float p = expf(sc[k] - mx);
    sc[k] = p;
    sum += p;
  }
  sum = wave_sum(sum);
  if (lane == 0) red[wave] = sum;
  __syncthreads();
  const float inv = 1.0f / (red[0] + red[1] + red[2] + red[3]);

  // probability-weighted values
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  for (int g0 = 0; g0 < n; g0 += 128) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      int key = g0 + u * 32 + wave * 8 + sub;
      if (key < n) {
        const T* vp = (SELF && key == n - 1) ? (srow + 2 * d) : (vb + (int64_t)key * 64);
        float vv[8];
        load8(vp + dc, vv);
        float p = sc[key];
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = fmaf(p, vv[i], acc[i]);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float a = acc[i];
    a += __shfl_xor(a, 8, 64);
    a += __shfl_xor(a, 16, 64);
    a += __shfl_xor(a, 32, 64);
    acc[i] = a;
  }
  if (lane < 8) {
#pragma unroll
    for (int i = 0; i < 8; ++i) ored[wave][dc + i] = acc[i];
  }
  __syncthreads();
  if (tid < 64) {
    float v = ored[0][tid] + ored[1][tid] + ored[2][tid] + ored[3][tid];
    St<T>::st(out, (int64_t)row * d + h * 64 + tid, v * inv);
  }
}

template <typename T>
void decode_self_attn(const T* qkv, T* cache, int64_t slot_stride, int64_t layer_off,
                      const int32_t* slots, const int32_t* pos, int D, int n_head, T* out,
                      hipStream_t s) {
  if (D > 0)
    k_decode_attn<T, true><<<dim3(n_head, D), 256, 0, s>>>(qkv, cache, slot_stride, layer_off,
                                                           slots, pos, n_head, out);
}
template <typename T>
void decode_cross_attn(const T* q, T* cache, int64_t slot_stride, int64_t layer_off,
                       const int32_t* slots, int D, int n_head, T* out, hipStream_t s) {
  if (D > 0)
    k_decode_attn<T, false><<<dim3(n_head, D), 256, 0, s>>>(q, cache, slot_stride, layer_off,
                                                            slots, nullptr, n_head, out);
}
template void decode_self_attn<float>(const float*, float*, int64_t, int64_t, const int32_t*,
                                      const int32_t*, int, int, float*, hipStream_t);
template void decode_self_attn<bf16_t>(const bf16_t*, bf16_t*, int64_t, int64_t, const int32_t*,
                                       const int32_t*, int, int, bf16_t*, hipStream_t);
template void decode_cross_attn<float>(const float*, float*, int64_t, int64_t, const int32_t*,
                                       int, int, float*, hipStream_t);
template void decode_cross_attn<bf16_t>(const bf16_t*, bf16_t*, int64_t, int64_t,
                                        const int32_t*, int, int, bf16_t*, hipStream_t);

}  // namespace asr
