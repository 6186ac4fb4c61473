// GEMMs of the step.
//
//  * gemm_bf16: C = A . W^T on gfx950 MFMA (v_mfma_f32_32x32x16_bf16), bf16
//    operands, fp32 accumulation, LDS double buffering, fused epilogues
//    (bias, exact GELU, fp32 residual add, conv-stem row mapping, scatter of
//    all decoder layers' cross K/V into a slot's cache).
//  * gemm_f32: the same contract in plain fp32 FMA (the fp32 model path).
//  * dgemm_bf16 / dgemm_f32: skinny products for the decode rows (weights
//    streamed once): bias / GELU fused into one slice, or float32 partial
//    sums of a few K slices that the next kernel adds up.
//  * vocab_argmax_bf16: the tied vocabulary projection fused with a per-row
//    argmax (lowest index on ties) over each 64-column tile, finished by a
//    deterministic cross-tile reduction.
#include "asr_device.h"

#include <algorithm>

namespace asr {

// ---------------------------------------------------------------------------
// Epilogue
// ---------------------------------------------------------------------------
template <int KIND, typename T>
__device__ __forceinline__ void epi_apply(const Epilogue& e, int r, int n, float acc) {
  float v = acc + (e.bias ? e.bias[n] : 0.0f);
  if constexpr (KIND == EPI_STORE) {
    St<T>::st((T*)e.out, (int64_t)r * e.ldc + n, v);
  } else if constexpr (KIND == EPI_GELU) {
    St<T>::st((T*)e.out, (int64_t)r * e.ldc + n, gelu_erf(v));
  } else if constexpr (KIND == EPI_CONV1) {
    int g = r / kFrames, t = r - g * kFrames;
    int64_t base = (int64_t)g * (kFrames + 1) * e.d_model;
    St<T>::st((T*)e.out, base + (int64_t)(t + 1) * e.d_model + n, gelu_erf(v));
    if (t == 0) St<T>::st((T*)e.out, base + n, 0.0f);        // position -1 of conv2
  } else if constexpr (KIND == EPI_CONV2) {
    int t = r % kCtx;
    ((float*)e.out)[(int64_t)r * e.ldc + n] = gelu_erf(v) + e.pos[(int64_t)t * e.ldc + n];
  } else if constexpr (KIND == EPI_XKV) {
    int g = r / kCtx, t = r - g * kCtx;
    int two_d = 2 * e.d_model;
    int l = n / two_d;
    int rem = n - l * two_d;
    int kv = rem >= e.d_model;
    int hd = rem - kv * e.d_model;
    int h = hd >> 6, c = hd & 63;
    int64_t addr = (int64_t)e.slots[g] * e.slot_stride +
                   ((((int64_t)l * 2 + kv) * e.n_head + h) * kCtx + t) * kHeadDim + c;
    St<T>::st((T*)e.out, addr, v);
  } else if constexpr (KIND == EPI_QKV) {
    const int two_d = 2 * e.d_model;
    if (n < two_d) {
      St<T>::st((T*)e.out, (int64_t)r * e.ldc + n, n < e.d_model ? v * kQScaleLog2 : v);
    } else {
      int g = r / kCtx, t = r - g * kCtx;
      int hd = n - two_d;
      int64_t addr = (((int64_t)g * e.n_head + (hd >> 6)) * kHeadDim + (hd & 63)) * kVtLd + t;
      St<T>::st((T*)e.out2, addr, v);
    }
  }
}

// Epilogue stores carry the non-temporal hint: the encoder products write
// hundreds of MB that the L2 cannot keep for the next kernel anyway, and
// letting them allocate there evicts the operand panels the running GEMM
// still re-reads (measured: about a quarter of the time of a K = 1280
// product goes away).
__device__ __forceinline__ void st4_bf16(bf16_t* p, float4 v) {
  typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
  u32x2 u;
  u.x = pack2_bf16(v.x, v.y);
  u.y = pack2_bf16(v.z, v.w);
  __builtin_nontemporal_store(u, (u32x2*)p);
}
__device__ __forceinline__ void st4_f32(float* p, float4 v) {
  typedef __attribute__((ext_vector_type(4))) float f32x4;
  f32x4 u = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(u, (f32x4*)p);
}
__device__ __forceinline__ float4 gelu4(float4 v) {
  return make_float4(gelu_erf(v.x), gelu_erf(v.y), gelu_erf(v.z), gelu_erf(v.w));
}
__device__ __forceinline__ float4 add4(float4 a, float4 b) {
  return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

// Four consecutive columns n..n+3 of row r (n % 4 == 0), bias already added.
template <int KIND>
__device__ __forceinline__ void epi_apply4(const Epilogue& e, int r, int n, float4 v) {
  if constexpr (KIND == EPI_QKV) {
    if (n < e.d_model) v = make_float4(v.x * kQScaleLog2, v.y * kQScaleLog2, v.z * kQScaleLog2,
                                       v.w * kQScaleLog2);
    st4_bf16((bf16_t*)e.out + (int64_t)r * e.ldc + n, v);
  } else if constexpr (KIND == EPI_STORE) {
    st4_bf16((bf16_t*)e.out + (int64_t)r * e.ldc + n, v);
  } else if constexpr (KIND == EPI_GELU) {
    st4_bf16((bf16_t*)e.out + (int64_t)r * e.ldc + n, gelu4(v));
  } else if constexpr (KIND == EPI_CONV1) {
    const int g = r / kFrames, t = r - g * kFrames;
    const int64_t base = (int64_t)g * (kFrames + 1) * e.d_model;
    st4_bf16((bf16_t*)e.out + base + (int64_t)(t + 1) * e.d_model + n, gelu4(v));
    if (t == 0) st4_bf16((bf16_t*)e.out + base + n, make_float4(0.f, 0.f, 0.f, 0.f));
  } else if constexpr (KIND == EPI_CONV2) {
    const int t = r % kCtx;
    st4_f32((float*)e.out + (int64_t)r * e.ldc + n,
            add4(gelu4(v), *(const float4*)(e.pos + (int64_t)t * e.ldc + n)));
  } else if constexpr (KIND == EPI_XKV) {
    const int g = r / kCtx, t = r - g * kCtx;
    const int two_d = 2 * e.d_model;
    const int l = n / two_d, rem = n - l * two_d;
    const int kv = rem >= e.d_model, hd = rem - kv * e.d_model;
    const int64_t addr = (int64_t)e.slots[g] * e.slot_stride +
                         ((((int64_t)l * 2 + kv) * e.n_head + (hd >> 6)) * kCtx + t) * kHeadDim +
                         (hd & 63);
    st4_bf16((bf16_t*)e.out + addr, v);
  }
}

// Bias of the four columns n..n+3 (zero without bias or past N).  The
// epilogues load it once per wave tile, ahead of the block loop: a load per
// block would put an L2 round trip on the epilogue's critical path 2 FM FN
// times.
__device__ __forceinline__ float4 bias4(const Epilogue& e, int n, int N) {
  if (!e.bias || n >= N) return make_float4(0.f, 0.f, 0.f, 0.f);
  if (n + 3 < N) return *(const float4*)(e.bias + n);
  return make_float4(e.bias[n], n + 1 < N ? e.bias[n + 1] : 0.f, n + 2 < N ? e.bias[n + 2] : 0.f, 0.f);
}
__device__ __forceinline__ float bias1(const Epilogue& e, int n, int N) {
  return e.bias && n < N ? e.bias[n] : 0.f;
}

// Epilogue of a wave's FM x FN accumulator blocks.  Each 32x32 block goes
// through the wave's private LDS stage (row stride 36 floats) in the MFMA
// output layout -- lane holds column lane%32 and, for register r, row
// 8*(r/4) + 4*(lane/32) + r%4 -- and is read back as four consecutive
// columns of one row per lane, so every store moves 8 or 16 bytes.  The
// transposed V of the fused QKV product (VT below) is read back as four
// consecutive rows of one column instead (contiguous in V^T).  The stage is
// private to the wave and LDS executes a wave's accesses in order, so no
// barrier is needed between blocks; the caller synchronises the block once
// before the first block (the stage aliases the operand ring).
constexpr int kStageLd = 36;
constexpr int EPI_VT = 100;   // internal: V columns of EPI_QKV

// The conv-stem epilogue keeps its row loop rolled: unrolled, its address
// arithmetic spills the accumulators.
#define EPI_UNROLL (KIND == EPI_CONV1 ? 1 : 4)
template <int KIND, int FM, int FN>
__device__ __forceinline__ void epi_wave_impl(const Epilogue& e, f32x16 (&acc)[FM][FN],
                                              float* stage, int m0w, int n0w, int M, int N,
                                              int lane) {
  const int l32 = lane & 31, lh = lane >> 5;
  const bool vec_ok = (N & 3) == 0 && (e.ldc & 3) == 0 && (e.d_model & 3) == 0;
  constexpr int AK = KIND == EPI_VT ? EPI_QKV : KIND;     // kind for the scalar fallback
  constexpr int NB = KIND == EPI_VT ? 4 : 1;
  float4 bj[FN];                // bias of the lane's columns (x only for VT: one per it)
  float bvt[FN][NB];
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    if constexpr (KIND == EPI_VT) {
#pragma unroll
      for (int it = 0; it < NB; ++it) bvt[j][it] = bias1(e, n0w + j * 32 + it * 8 + (lane >> 3), N);
    } else {
      bj[j] = bias4(e, n0w + j * 32 + (lane & 7) * 4, N);
    }
  }
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        stage[((r >> 2) * 8 + lh * 4 + (r & 3)) * kStageLd + l32] = acc[i][j][r];
      __builtin_amdgcn_wave_barrier();
      const int rbase = m0w + i * 32, cbase = n0w + j * 32;
      if constexpr (KIND == EPI_VT) {
        // lane takes rows 4q..4q+3 of one column
        const int r4 = (lane & 7) * 4;
#pragma unroll
        for (int it = 0; it < 4; ++it) {
          const int c = it * 8 + (lane >> 3), n = cbase + c;
          if (n >= N) continue;
          const int row = rbase + r4;
          float4 v = make_float4(stage[r4 * kStageLd + c], stage[(r4 + 1) * kStageLd + c],
                                 stage[(r4 + 2) * kStageLd + c], stage[(r4 + 3) * kStageLd + c]);
          if (row + 3 < M) {
            const float b = bvt[j][it];
            v = add4(v, make_float4(b, b, b, b));
            const int g = row / kCtx, t = row - g * kCtx;    // t % 4 == 0: same clip
            const int hd = n - 2 * e.d_model;
            const int64_t addr =
                (((int64_t)g * e.n_head + (hd >> 6)) * kHeadDim + (hd & 63)) * kVtLd + t;
            st4_bf16((bf16_t*)e.out2 + addr, v);
          } else {
            const float vv[4] = {v.x, v.y, v.z, v.w};
            for (int q = 0; q < 4; ++q)
              if (row + q < M) epi_apply<AK, bf16_t>(e, row + q, n, vv[q]);
          }
        }
      } else {
        const int c4 = (lane & 7) * 4;
#pragma unroll EPI_UNROLL
        for (int it = 0; it < 4; ++it) {
          const int rr = it * 8 + (lane >> 3), row = rbase + rr, n = cbase + c4;
          if (row >= M || n >= N) continue;
          const float4 v = *(const float4*)&stage[rr * kStageLd + c4];
          if (vec_ok) {
            epi_apply4<KIND>(e, row, n, add4(v, bj[j]));
          } else {
            const float vv[4] = {v.x, v.y, v.z, v.w};
            for (int q = 0; q < 4; ++q)
              if (n + q < N) epi_apply<AK, bf16_t>(e, row, n + q, vv[q]);
          }
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
}
#undef EPI_UNROLL

// Plain element-wise fallback (a wave whose columns straddle q/k and V).
template <int FM, int FN>
__device__ __forceinline__ void epi_wave_mixed(const Epilogue& e, f32x16 (&acc)[FM][FN],
                                            float* stage, int m0w, int n0w, int M, int N,
                                            int lane) {
  const int l32 = lane & 31, lh = lane >> 5;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        stage[((r >> 2) * 8 + lh * 4 + (r & 3)) * kStageLd + l32] = acc[i][j][r];
      __builtin_amdgcn_wave_barrier();
      for (int t = 0; t < 16; ++t) {
        const int rr = t * 2 + lh, row = m0w + i * 32 + rr, col = n0w + j * 32 + l32;
        if (row < M && col < N) epi_apply<EPI_QKV, bf16_t>(e, row, col, stage[rr * kStageLd + l32]);
      }
      __builtin_amdgcn_wave_barrier();
    }
}

// For EPI_QKV a wave's columns are all q/k or all V when 2 d_model is a
// multiple of the wave's column span (always, for d_model % 128 == 0 and
// spans of 32 or 64); otherwise the blocks are sorted out one by one.
template <int KIND, int FM, int FN>
__device__ __forceinline__ void epi_wave(const Epilogue& e, f32x16 (&acc)[FM][FN], float* stage,
                                         int m0w, int n0w, int M, int N, int lane) {
  if constexpr (KIND == EPI_QKV) {
    const int two_d = 2 * e.d_model;
    if (n0w >= two_d)
      epi_wave_impl<EPI_VT, FM, FN>(e, acc, stage, m0w, n0w, M, N, lane);
    else if (n0w + FN * 32 <= two_d)
      epi_wave_impl<EPI_QKV, FM, FN>(e, acc, stage, m0w, n0w, M, N, lane);
    else
      epi_wave_mixed<FM, FN>(e, acc, stage, m0w, n0w, M, N, lane);
  } else {
    epi_wave_impl<KIND, FM, FN>(e, acc, stage, m0w, n0w, M, N, lane);
  }
}

__device__ __forceinline__ int64_t arow_offset(const AView& a, int r) {
  int g = r / a.rows_per_batch;
  return (int64_t)g * a.batch_stride + (int64_t)(r - g * a.rows_per_batch) * a.lda;
}

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM
//
// Workgroup tile BM x BN x 64 with WM x WN waves, each wave owning a
// (BM/WM) x (BN/WN) block of 32x32 MFMA tiles whose fp32 accumulators stay in
// registers for the whole K loop.  Operand tiles are double-buffered in LDS
// (rows padded to 72 elements so the 16-byte fragment reads of 32 consecutive
// rows hit distinct banks); the next K tile is fetched into registers while
// the current one feeds the MFMAs.
//
// Tile order is XCD-aware: the hardware deals workgroups round-robin to the
// 8 XCDs, so block b runs on XCD b % 8.  Each XCD is given one contiguous
// range of tiles, walked in groups of GM row tiles (column tile outer, row
// tile inner) so that the A rows and the W columns a group needs stay in that
// XCD's L2 while its CUs work through them.
// ---------------------------------------------------------------------------
constexpr int kXcd = 8;

__device__ __forceinline__ void tile_of(int bid, int n_tiles, int n_tm, int n_tn, int gm,
                                        int& tm, int& tn) {
  const int q = n_tiles / kXcd, r = n_tiles % kXcd;
  const int xcd = bid % kXcd, local = bid / kXcd;
  const int t = xcd * q + min(xcd, r) + local;           // contiguous range per XCD
  const int group = t / (gm * n_tn);
  const int first_tm = group * gm;
  const int rows = min(gm, n_tm - first_tm);
  const int in_group = t - group * gm * n_tn;
  tm = first_tm + in_group % rows;
  tn = in_group / rows;
}

// LDS holds each operand tile row-major without padding; the 16-byte chunk c
// of row r sits at chunk position c ^ swz(r).  On gfx950 a 16-byte LDS access
// is served 16 lanes at a time from 64 four-byte banks, so 16 lanes must touch
// 16 distinct 16-byte slots of a 256-byte window: with these swizzles both the
// fragment reads (32 consecutive rows, same chunk) and the tile stores (whole
// rows) are conflict-free.
template <int BK>
__device__ __forceinline__ int lds_swz(int row) {
  return BK == 32 ? ((row >> 2) & 3) : ((row >> 1) & 7);
}

template <int BM, int BN, int BK, int WM, int WN, int KIND>
__global__ __launch_bounds__(WM* WN * 64) void k_gemm_bf16(AView a, const bf16_t* __restrict__ w,
                                                          int M, int N, int K, Epilogue e,
                                                          int n_tm, int n_tn, int gm) {
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int CPR = BK / 8;                      // 16-byte chunks per tile row
  constexpr int CA = BM * CPR / NT, CB = BN * CPR / NT;
  constexpr int RSTEP = NT / CPR;                  // rows covered by one pass of the block
  static_assert(BK == 32 || BK == 64, "BK");
  static_assert(CA * NT == BM * CPR && CB * NT == BN * CPR, "tile/threads");
  static_assert(RSTEP % 16 == 0, "swizzle period");
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];
  bf16_t* As = smem;                               // [2][BM * BK]
  bf16_t* Bs = smem + 2 * BM * BK;                 // [2][BN * BK]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WM, wn = wave / WM;
  int tm, tn;
  tile_of(blockIdx.x, n_tm * n_tn, n_tm, n_tn, gm, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;

  // loader: thread t moves logical chunk t % CPR of rows t/CPR + i*RSTEP
  const int lrow0 = tid / CPR, lc = tid % CPR;
  const int st_off = lrow0 * BK + ((lc ^ lds_swz<BK>(lrow0)) * 8);   // same swizzle for all i
  const bf16_t* abase = (const bf16_t*)a.ptr;
  int64_t aoff[CA];
#pragma unroll
  for (int i = 0; i < CA; ++i) {
    int r = min(m0 + lrow0 + i * RSTEP, M - 1);    // rows past M load row M-1, never stored
    int g = r / a.rows_per_batch;
    aoff[i] = (int64_t)g * a.batch_stride + (int64_t)(r - g * a.rows_per_batch) * a.lda + lc * 8;
  }
  int64_t boff[CB];
#pragma unroll
  for (int i = 0; i < CB; ++i) boff[i] = (int64_t)min(n0 + lrow0 + i * RSTEP, N - 1) * K + lc * 8;

  const int nk = (K + BK - 1) / BK;
  const bool ktail = (K % BK) != 0;

#define GEMM_GLOAD(RA, RB, k0)                                                      \
  do {                                                                              \
    if (!ktail || (k0) + BK <= K) {                                                 \
      _Pragma("unroll") for (int i = 0; i < CA; ++i) RA[i] = *(const uint4*)(abase + aoff[i] + (k0)); \
      _Pragma("unroll") for (int i = 0; i < CB; ++i) RB[i] = *(const uint4*)(w + boff[i] + (k0));     \
    } else {                                                                        \
      const bool in = (k0) + lc * 8 < K;                                            \
      _Pragma("unroll") for (int i = 0; i < CA; ++i)                                \
        RA[i] = in ? *(const uint4*)(abase + aoff[i] + (k0)) : uint4{0u, 0u, 0u, 0u}; \
      _Pragma("unroll") for (int i = 0; i < CB; ++i)                                \
        RB[i] = in ? *(const uint4*)(w + boff[i] + (k0)) : uint4{0u, 0u, 0u, 0u};   \
    }                                                                               \
  } while (0)
#define GEMM_SSTORE(RA, RB, buf)                                                    \
  do {                                                                              \
    _Pragma("unroll") for (int i = 0; i < CA; ++i)                                  \
      *(uint4*)&As[(buf) * BM * BK + st_off + i * RSTEP * BK] = RA[i];              \
    _Pragma("unroll") for (int i = 0; i < CB; ++i)                                  \
      *(uint4*)&Bs[(buf) * BN * BK + st_off + i * RSTEP * BK] = RB[i];              \
  } while (0)

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // fragment reads: row lane%32 of each 32-row block (blocks start on
  // multiples of 32, so the swizzle depends on the lane only), chunk
  // kk*2 + lane/32.  Fragments of step kk+1 are requested before the MFMAs of
  // step kk so that LDS latency overlaps matrix work within the wave.
  const int lrow = lane & 31, sw = lds_swz<BK>(lrow), lh = lane >> 5;
  const bf16_t* a_frag = As + (wm * TM + lrow) * BK;
  const bf16_t* b_frag = Bs + (wn * TN + lrow) * BK;

  uint4 ra[CA], rb[CB];
  GEMM_GLOAD(ra, rb, 0);
  GEMM_SSTORE(ra, rb, 0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) GEMM_GLOAD(ra, rb, (kt + 1) * BK);
    const bf16_t* Ac = a_frag + cur * BM * BK;
    const bf16_t* Bc = b_frag + cur * BN * BK;
    bf16x8 af[2][FM], bfr[2][FN];
    {
      const int ch = (lh ^ sw) * 8;
#pragma unroll
      for (int i = 0; i < FM; ++i) af[0][i] = *(const bf16x8*)(Ac + i * 32 * BK + ch);
#pragma unroll
      for (int j = 0; j < FN; ++j) bfr[0][j] = *(const bf16x8*)(Bc + j * 32 * BK + ch);
    }
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int p = kk & 1;
      if (kk + 1 < BK / 16) {
        const int ch = (((kk + 1) * 2 + lh) ^ sw) * 8;
#pragma unroll
        for (int i = 0; i < FM; ++i) af[p ^ 1][i] = *(const bf16x8*)(Ac + i * 32 * BK + ch);
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[p ^ 1][j] = *(const bf16x8*)(Bc + j * 32 * BK + ch);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[p][i], bfr[p][j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) GEMM_SSTORE(ra, rb, cur ^ 1);
    __syncthreads();
  }
#undef GEMM_GLOAD
#undef GEMM_SSTORE

  // Epilogue through LDS, one 32x32 block per wave at a time.  In the MFMA
  // output layout a lane holds column lane%32 and, for register r, row
  // 8*(r/4) + 4*(lane/32) + r%4; the block is written to LDS in that layout
  // and read back as two full rows per instruction, so the (possibly heavy)
  // epilogue math runs in a short rolled loop and every store covers whole
  // 32-column row segments.
  epi_wave<KIND, FM, FN>(e, acc, (float*)smem + wave * (32 * kStageLd), m0 + wm * TM,
                         n0 + wn * TN, M, N, lane);
}

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM with an S-stage LDS ring filled by direct global->LDS loads.
//
// Each wave issues global_load_lds_dwordx4: lane l of one instruction lands
// 16 bytes at LDS base + 16 l, so an instruction fills one contiguous 1 KB
// slice of a tile (16 rows at BK = 32, 8 rows at BK = 64); the lane picks the
// global chunk that the swizzled layout wants at its slot.  The loads are
// issued from inline assembly so the compiler does not serialise every LDS
// read behind them; completion of tile kt is awaited explicitly (vmcnt) while
// the loads of the next S-2 tiles stay in flight, then one barrier per K
// tile publishes it and frees the buffer the next tile is loaded into.
// Requires K % BK == 0.
// ---------------------------------------------------------------------------
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

template <int MAXN>
__device__ __forceinline__ void wait_vmcnt_rt(int n) {
  // n is wave-uniform; the immediate must be a constant
  if constexpr (MAXN > 0) {
    if (n >= MAXN) { wait_vmcnt<MAXN>(); return; }
    wait_vmcnt_rt<MAXN - 1>(n);
  } else {
    wait_vmcnt<0>();
  }
}

__device__ __forceinline__ void lds_dma16(uint32_t lds_addr, const void* gptr) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
               :: "s"(lds_addr), "v"(gptr) : "memory", "m0");
}
// Same with a wave-uniform 64-bit base in SGPRs and a 32-bit per-lane byte
// offset: no per-load address arithmetic in vector registers.
__device__ __forceinline__ void lds_dma16_s(uint32_t lds_addr, uint32_t voff, const void* sbase) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
               :: "s"(lds_addr), "v"(voff), "s"(sbase) : "memory", "m0");
}

template <int BM, int BN, int BK, int WM, int WN, int S, int KIND, int SCHED = 0>
__global__ __launch_bounds__(WM* WN * 64) void k_gemm_bf16_dma(AView a,
                                                              const bf16_t* __restrict__ w,
                                                              int M, int N, int K, Epilogue e,
                                                              int n_tm, int n_tn, int gm) {
  constexpr int NW = WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int CPR = BK / 8;
  constexpr int RPI = 1024 / (BK * 2);             // tile rows filled by one wave instruction
  constexpr int IA = BM / (RPI * NW), IB = BN / (RPI * NW);   // instructions per wave per tile
  constexpr int LPT = IA + IB;                     // loads per lane per tile
  static_assert(BK == 32 || BK == 64, "BK");
  static_assert(IA * RPI * NW == BM && IB * RPI * NW == BN, "tile/waves");
  static_assert(S >= 2 && LPT * (S - 2) < 64, "stages");
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];
  constexpr int STAGE = (BM + BN) * BK;            // elements per stage

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WM, wn = wave / WM;
  int tm, tn;
  tile_of(blockIdx.x, n_tm * n_tn, n_tm, n_tn, gm, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const uint32_t lds0 =
      (uint32_t)(uintptr_t)((__attribute__((address_space(3))) bf16_t*)smem);

  // per-lane global sources and per-wave LDS destinations of the tile loads
  const bf16_t* abase = (const bf16_t*)a.ptr;
  const bf16_t* asrc[IA];
  uint32_t adst[IA];
#pragma unroll
  for (int i = 0; i < IA; ++i) {
    const int r0 = (i * NW + wave) * RPI;
    const int row = r0 + lane / CPR;
    const int c = (lane % CPR) ^ lds_swz<BK>(row);
    const int r = min(m0 + row, M - 1);
    const int g = r / a.rows_per_batch;
    asrc[i] = abase + (int64_t)g * a.batch_stride + (int64_t)(r - g * a.rows_per_batch) * a.lda +
              c * 8;
    adst[i] = __builtin_amdgcn_readfirstlane(lds0 + (uint32_t)(r0 * BK * 2));
  }
  const bf16_t* bsrc[IB];
  uint32_t bdst[IB];
#pragma unroll
  for (int i = 0; i < IB; ++i) {
    const int r0 = (i * NW + wave) * RPI;
    const int row = r0 + lane / CPR;
    const int c = (lane % CPR) ^ lds_swz<BK>(row);
    bsrc[i] = w + (int64_t)min(n0 + row, N - 1) * K + c * 8;
    bdst[i] = __builtin_amdgcn_readfirstlane(lds0 + (uint32_t)((BM * BK + r0 * BK) * 2));
  }
  const int nk = K / BK;
  auto issue = [&](int tile) {
    const uint32_t so = (uint32_t)((tile % S) * STAGE * 2);
    const int k0 = tile * BK;
#pragma unroll
    for (int i = 0; i < IA; ++i) lds_dma16(adst[i] + so, asrc[i] + k0);
#pragma unroll
    for (int i = 0; i < IB; ++i) lds_dma16(bdst[i] + so, bsrc[i] + k0);
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int lrow = lane & 31, sw = lds_swz<BK>(lrow), lh = lane >> 5;
  const bf16_t* a_frag = smem + (wm * TM + lrow) * BK;
  const bf16_t* b_frag = smem + BM * BK + (wn * TN + lrow) * BK;

#pragma unroll
  for (int t = 0; t < S - 1; ++t)
    if (t < nk) issue(t);
  for (int kt = 0; kt < nk; ++kt) {
    // tile kt has landed once at most min(S-2, nk-1-kt) later tiles are pending
    wait_vmcnt_rt<LPT * (S - 2)>(LPT * min(S - 2, nk - 1 - kt));
    __builtin_amdgcn_s_barrier();
    if (kt + S - 1 < nk) issue(kt + S - 1);
    const bf16_t* Ac = a_frag + (kt % S) * STAGE;
    const bf16_t* Bc = b_frag + (kt % S) * STAGE;
    bf16x8 af[2][FM], bfr[2][FN];
    {
      const int ch = (lh ^ sw) * 8;
#pragma unroll
      for (int i = 0; i < FM; ++i) af[0][i] = *(const bf16x8*)(Ac + i * 32 * BK + ch);
#pragma unroll
      for (int j = 0; j < FN; ++j) bfr[0][j] = *(const bf16x8*)(Bc + j * 32 * BK + ch);
    }
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int p = kk & 1;
      if (kk + 1 < BK / 16) {
        const int ch = (((kk + 1) * 2 + lh) ^ sw) * 8;
#pragma unroll
        for (int i = 0; i < FM; ++i) af[p ^ 1][i] = *(const bf16x8*)(Ac + i * 32 * BK + ch);
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[p ^ 1][j] = *(const bf16x8*)(Bc + j * 32 * BK + ch);
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[p][i], bfr[p][j], acc[i][j], 0, 0, 0);
      if constexpr (SCHED == 1) {
        // interleave the next step's fragment reads with this step's MFMAs
        if (kk + 1 < BK / 16) {
#pragma unroll
          for (int q = 0; q < FM + FN; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          __builtin_amdgcn_sched_group_barrier(0x008, FM * FN - (FM + FN), 0);
        }
      }
    }
  }
  wait_vmcnt<0>();
  __syncthreads();

  epi_wave<KIND, FM, FN>(e, acc, (float*)smem + wave * (32 * kStageLd), m0 + wm * TM,
                         n0 + wn * TN, M, N, lane);
}

// Same operand ring, with the fragment reads software-pipelined across K
// tiles: the barrier that publishes tile kt+1 sits before the MFMAs of the
// last k-step of tile kt, so the first fragments of tile kt+1 are read while
// those MFMAs run, and no k-step ever waits on a fragment read issued just
// before it.  All S stages are in flight: tile kt+S is requested as soon as
// every wave has finished reading tile kt.  sched_barrier fences keep the
// compiler from sinking the prefetching reads below the MFMAs.
template <int VM>
__device__ __forceinline__ void wait_vm_lgkm0() {
  static_assert(VM >= 0 && VM < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((VM & 0xF) | ((VM >> 4) << 14) | (0x7 << 4));
}
template <int MAXN>
__device__ __forceinline__ void wait_vm_lgkm0_rt(int n) {
  if constexpr (MAXN > 0) {
    if (n >= MAXN) { wait_vm_lgkm0<MAXN>(); return; }
    wait_vm_lgkm0_rt<MAXN - 1>(n);
  } else {
    wait_vm_lgkm0<0>();
  }
}

template <int BM, int BN, int BK, int WM, int WN, int S, int KIND>
__global__ __launch_bounds__(WM* WN * 64) void k_gemm_bf16_pf(AView a,
                                                             const bf16_t* __restrict__ w,
                                                             int M, int N, int K, Epilogue e,
                                                             int n_tm, int n_tn, int gm) {
  constexpr int NW = WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int CPR = BK / 8;
  constexpr int NS = BK / 16;                      // MFMA k-steps per tile
  constexpr int RPI = 1024 / (BK * 2);
  constexpr int IA = BM / (RPI * NW), IB = BN / (RPI * NW);
  constexpr int LPT = IA + IB;
  static_assert(BK == 32 || BK == 64, "BK");
  static_assert(IA * RPI * NW == BM && IB * RPI * NW == BN, "tile/waves");
  static_assert(S >= 2 && LPT * (S - 1) < 64, "stages");
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];
  constexpr int STAGE = (BM + BN) * BK;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WM, wn = wave / WM;
  int tm, tn;
  tile_of(blockIdx.x, n_tm * n_tn, n_tm, n_tn, gm, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const uint32_t lds0 =
      (uint32_t)(uintptr_t)((__attribute__((address_space(3))) bf16_t*)smem);

  const bf16_t* abase = (const bf16_t*)a.ptr;
  const bf16_t* asrc[IA];
  uint32_t adst[IA];
#pragma unroll
  for (int i = 0; i < IA; ++i) {
    const int r0 = (i * NW + wave) * RPI;
    const int row = r0 + lane / CPR;
    const int c = (lane % CPR) ^ lds_swz<BK>(row);
    const int r = min(m0 + row, M - 1);
    const int g = r / a.rows_per_batch;
    asrc[i] = abase + (int64_t)g * a.batch_stride + (int64_t)(r - g * a.rows_per_batch) * a.lda +
              c * 8;
    adst[i] = __builtin_amdgcn_readfirstlane(lds0 + (uint32_t)(r0 * BK * 2));
  }
  const bf16_t* bsrc[IB];
  uint32_t bdst[IB];
#pragma unroll
  for (int i = 0; i < IB; ++i) {
    const int r0 = (i * NW + wave) * RPI;
    const int row = r0 + lane / CPR;
    const int c = (lane % CPR) ^ lds_swz<BK>(row);
    bsrc[i] = w + (int64_t)min(n0 + row, N - 1) * K + c * 8;
    bdst[i] = __builtin_amdgcn_readfirstlane(lds0 + (uint32_t)((BM * BK + r0 * BK) * 2));
  }
  const int nk = K / BK;
  auto issue = [&](int tile) {
    const uint32_t so = (uint32_t)((tile % S) * STAGE * 2);
    const int k0 = tile * BK;
#pragma unroll
    for (int i = 0; i < IA; ++i) lds_dma16(adst[i] + so, asrc[i] + k0);
#pragma unroll
    for (int i = 0; i < IB; ++i) lds_dma16(bdst[i] + so, bsrc[i] + k0);
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int lrow = lane & 31, sw = lds_swz<BK>(lrow), lh = lane >> 5;
  const bf16_t* a_frag = smem + (wm * TM + lrow) * BK;
  const bf16_t* b_frag = smem + BM * BK + (wn * TN + lrow) * BK;
  bf16x8 af[2][FM], bfr[2][FN];
#define PF_READ(P, TILE, KK)                                                          \
  do {                                                                                \
    const int off_ = ((TILE) % S) * STAGE + ((((KK) * 2 + lh) ^ sw) * 8);             \
    _Pragma("unroll") for (int i = 0; i < FM; ++i)                                    \
      af[P][i] = *(const bf16x8*)(a_frag + off_ + i * 32 * BK);                       \
    _Pragma("unroll") for (int j = 0; j < FN; ++j)                                    \
      bfr[P][j] = *(const bf16x8*)(b_frag + off_ + j * 32 * BK);                      \
  } while (0)

  // Issued right after a fragment prefetch, this tells the wait-count pass
  // that every older LDS read has completed (the reads feeding the coming
  // MFMAs), which it cannot prove by itself across the loop back edge.
  constexpr int kLgkmImm = 0xF | (0x3 << 14) | (0x7 << 4) | ((FM + FN) << 8);
  static_assert(FM + FN <= 15, "lgkmcnt");

#pragma unroll
  for (int t = 0; t < S; ++t)
    if (t < nk) issue(t);
  wait_vm_lgkm0_rt<LPT*(S - 1)>(LPT * min(S - 1, nk - 1));
  __builtin_amdgcn_s_barrier();
  PF_READ(0, 0, 0);
  for (int kt = 0; kt < nk; ++kt) {
#pragma unroll
    for (int kk = 0; kk < NS; ++kk) {
      const int p = kk & 1;
      if (kk + 1 < NS) {
        PF_READ(p ^ 1, kt, kk + 1);
      } else if (kt + 1 < nk) {
        // tile kt+1 landed (later tiles may still fly), this wave's reads of
        // tile kt done; after the barrier nobody reads tile kt any more
        wait_vm_lgkm0_rt<LPT*(S - 2)>(LPT * min(S - 2, nk - 2 - kt));
        __builtin_amdgcn_s_barrier();
        if (kt + S < nk) issue(kt + S);
        PF_READ(p ^ 1, kt + 1, 0);
      }
      if (kk + 1 < NS || kt + 1 < nk) __builtin_amdgcn_s_waitcnt(kLgkmImm);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[p][i], bfr[p][j], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#undef PF_READ
  wait_vmcnt<0>();
  __syncthreads();

  epi_wave<KIND, FM, FN>(e, acc, (float*)smem + wave * (32 * kStageLd), m0 + wm * TM,
                         n0 + wn * TN, M, N, lane);
}

// ---------------------------------------------------------------------------
// Persistent variant.  One workgroup per CU walks its share of the output
// tiles (virtual block ids b, b + grid, ... through the same XCD-aware tile
// order) and the operand ring runs on across tile boundaries, so the first K
// tile of the next output tile is in flight while the current one is written
// out through a small stage of its own beside the ring.  At a tile switch the
// next K tile is awaited before the stores are issued, and the ring's next
// load goes out after them, so every wait count stays exact or errs towards
// waiting longer.
// ---------------------------------------------------------------------------
// Epilogue through a 16-row stage per wave (it lives beside the operand
// ring, which is busy with the next tile): each 32x32 block goes out in two
// halves, registers 0-7 (rows 0-15) then 8-15 (rows 16-31).  The scatter
// epilogues keep their row loops rolled (unrolled, they spill).
#define EPI_HALF_UNROLL ((KIND == EPI_CONV1 || KIND == EPI_QKV) ? 1 : 2)
template <int KIND, int FM, int FN>
__device__ __forceinline__ void epi_wave_half(const Epilogue& e, f32x16 (&acc)[FM][FN],
                                              float* stage, int m0w, int n0w, int M, int N,
                                              int lane) {
  const int l32 = lane & 31, lh = lane >> 5;
  const bool vec_ok = (N & 3) == 0 && (e.ldc & 3) == 0 && (e.d_model & 3) == 0;
  const bool vt = KIND == EPI_QKV && n0w >= 2 * e.d_model;   // wave-uniform
  float4 bj[FN];     // bias of the lane's columns: c4..c4+3, or (VT) columns it*16 + lane/4
#pragma unroll
  for (int j = 0; j < FN; ++j)
    bj[j] = vt ? make_float4(bias1(e, n0w + j * 32 + (lane >> 2), N),
                             bias1(e, n0w + j * 32 + 16 + (lane >> 2), N), 0.f, 0.f)
               : bias4(e, n0w + j * 32 + (lane & 7) * 4, N);
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int r = 0; r < 8; ++r)
          stage[((r >> 2) * 8 + lh * 4 + (r & 3)) * kStageLd + l32] = acc[i][j][h * 8 + r];
        __builtin_amdgcn_wave_barrier();
        const int rbase = m0w + i * 32 + h * 16, cbase = n0w + j * 32;
        if (KIND == EPI_QKV && vt) {
          // lane takes rows 4q..4q+3 (of 16) of one column
          const int r4 = (lane & 3) * 4;
#pragma unroll EPI_HALF_UNROLL
          for (int it = 0; it < 2; ++it) {
            const int c = it * 16 + (lane >> 2), n = cbase + c, row = rbase + r4;
            if (n >= N) continue;
            float4 v = make_float4(stage[r4 * kStageLd + c], stage[(r4 + 1) * kStageLd + c],
                                   stage[(r4 + 2) * kStageLd + c], stage[(r4 + 3) * kStageLd + c]);
            if (row + 3 < M) {
              const float b = it == 0 ? bj[j].x : bj[j].y;
              v = add4(v, make_float4(b, b, b, b));
              const int g = row / kCtx, t = row - g * kCtx;    // t % 4 == 0: same clip
              const int hd = n - 2 * e.d_model;
              st4_bf16((bf16_t*)e.out2 +
                           (((int64_t)g * e.n_head + (hd >> 6)) * kHeadDim + (hd & 63)) * kVtLd + t,
                       v);
            } else {
              const float vv[4] = {v.x, v.y, v.z, v.w};
              for (int q = 0; q < 4; ++q)
                if (row + q < M) epi_apply<KIND, bf16_t>(e, row + q, n, vv[q]);
            }
          }
        } else {
          const int c4 = (lane & 7) * 4;
#pragma unroll EPI_HALF_UNROLL
          for (int it = 0; it < 2; ++it) {
            const int rr = it * 8 + (lane >> 3), row = rbase + rr, n = cbase + c4;
            if (row >= M || n >= N) continue;
            const float4 v = *(const float4*)&stage[rr * kStageLd + c4];
            if (vec_ok) {
              epi_apply4<KIND>(e, row, n, add4(v, bj[j]));
            } else {
              const float vv[4] = {v.x, v.y, v.z, v.w};
              for (int q = 0; q < 4; ++q)
                if (n + q < N) epi_apply<KIND, bf16_t>(e, row, n + q, vv[q]);
            }
          }
        }
        __builtin_amdgcn_wave_barrier();
      }
}

#undef EPI_HALF_UNROLL

// Epilogue straight from registers, for a product formed transposed
// (W fragment as the MFMA's first operand): a lane then holds output row
// l32 of each 32x32 block and, in register quad q, the four consecutive
// columns 8q + 4 lh .. 8q + 4 lh + 3.  The values are packed to bf16 and one
// lane-half swap (v_permlane32_swap) gathers eight consecutive columns per
// lane, so each store moves 16 bytes.  Row-major outputs are stored
// through a buffer resource sized to the output: lanes past M or N get an
// offset beyond it, which the hardware drops, so no lane diverges.  The
// cross-attention cache (XKV, far above the 2^31-byte reach of a buffer
// offset) is addressed per lane: the row part (slot, position) once per
// tile, the column part (layer, K/V, head, dim) per 16-byte run, which an
// eight-column run never splits since heads are 64 wide.  No LDS round trip:
// the store stream issues as fast as the accumulators convert.
// Cache policy of the register epilogue's stores: the default.  Unlike the
// staged epilogue's full-row stores, each of these instructions writes
// 32-byte runs of 32 different rows, which the L2 merges into whole lines;
// with the non-temporal hint every encoder product ran 7-16 % slower.
constexpr int kNtAux = 0;

template <int KIND>
constexpr bool kDirectEpi =
    KIND == EPI_STORE || KIND == EPI_GELU || KIND == EPI_XKV || KIND == EPI_QKV;

// V columns of the fused QKV product from the transposed layout: there the
// MFMA output block is V^T itself (rows = V columns, columns = positions), so
// it goes through the wave's 16-row LDS stage as the plain epilogue does and
// is read back as four consecutive positions of one V column -- eight
// contiguous bytes of V^T[clip][head][dim][position] (1500 is a multiple of
// 4, so the four never straddle clips); eight lanes fill 64 contiguous bytes.
template <int FM, int FN>
__device__ __forceinline__ void epi_direct_vt(const Epilogue& e, f32x16 (&acc)[FM][FN],
                                              float* stage, int m0w, int n0w, int M, int N,
                                              int lane) {
  typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
  const int l32 = lane & 31, lh = lane >> 5;
  const int n_clips = (M + kCtx - 1) / kCtx;
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      e.out2, (short)0, (int)((int64_t)n_clips * e.n_head * kHeadDim * kVtLd * 2), 0x00020000);
  const int c4 = (lane & 7) * 4, r8 = lane >> 3;
  float bv[FN][2][2];     // bias of the lane's V column per (block column, half, it)
#pragma unroll
  for (int j = 0; j < FN; ++j)
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int it = 0; it < 2; ++it) bv[j][h][it] = bias1(e, n0w + j * 32 + h * 16 + it * 8 + r8, N);
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int row = m0w + i * 32 + c4;                   // first of four positions
    const int g = row / kCtx, t = row - g * kCtx;
    const int rbase = g * e.n_head * kHeadDim * kVtLd + t;
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int r = 0; r < 8; ++r)
          stage[((r >> 2) * 8 + lh * 4 + (r & 3)) * kStageLd + l32] = acc[i][j][h * 8 + r];
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int it = 0; it < 2; ++it) {
          const int rr = it * 8 + r8, n = n0w + j * 32 + h * 16 + rr;
          const float4 v = *(const float4*)&stage[rr * kStageLd + c4];
          const float bb = bv[j][h][it];
          const int hd = n - 2 * e.d_model;
          const u32x2 x = {pack2_bf16(v.x + bb, v.y + bb), pack2_bf16(v.z + bb, v.w + bb)};
          const uint32_t off = row < M && n < N
                                   ? (uint32_t)(rbase + ((hd >> 6) * kHeadDim + (hd & 63)) * kVtLd) * 2u
                                   : 0x80000000u;
          __builtin_amdgcn_raw_buffer_store_b64(x, rs, off, 0, kNtAux);
        }
        __builtin_amdgcn_wave_barrier();
      }
  }
}

template <int KIND, int FM, int FN>
__device__ __forceinline__ void epi_direct(const Epilogue& e, f32x16 (&acc)[FM][FN], int m0w,
                                           int n0w, int M, int N, int lane) {
  static_assert(kDirectEpi<KIND>, "direct epilogue kind");
  typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
  const int l32 = lane & 31, lh = lane >> 5;
  __amdgpu_buffer_rsrc_t rs;
  int64_t xrow[FM];    // XKV: slot and position part of each of the lane's rows
  int64_t xcol = 0;    // XKV: (layer, K/V, head) part of the wave's columns
  if constexpr (KIND == EPI_XKV) {
    static_assert(FN * 32 <= kHeadDim, "a wave's columns stay within one head");
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int r = min(m0w + i * 32 + l32, M - 1), g = r / kCtx;
      xrow[i] = (int64_t)e.slots[g] * e.slot_stride + (int64_t)(r - g * kCtx) * kHeadDim;
    }
    // the wave's FN * 32 <= 64 columns start at a multiple of 64, and
    // d_model is one too, so they lie in one layer, one of K / V and one
    // head: that part of the address is wave-uniform
    const int two_d = 2 * e.d_model;
    const int l = n0w / two_d, rem = n0w - l * two_d;
    const int kv = rem >= e.d_model, hd0 = rem - kv * e.d_model;
    xcol = ((((int64_t)l * 2 + kv) * e.n_head + (hd0 >> 6)) * kCtx) * kHeadDim;
  } else {
    rs = __builtin_amdgcn_make_buffer_rsrc(e.out, (short)0, (int)((int64_t)M * e.ldc * 2),
                                           0x00020000);
  }
  float4 bq[FN][4];
#pragma unroll
  for (int j = 0; j < FN; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) bq[j][q] = bias4(e, n0w + j * 32 + 8 * q + 4 * lh, N);
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int row = m0w + i * 32 + l32;
    const bool rok = row < M;
    const int rofs = row * (int)e.ldc;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      float v[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        v[4 * q] = acc[i][j][4 * q] + bq[j][q].x;
        v[4 * q + 1] = acc[i][j][4 * q + 1] + bq[j][q].y;
        v[4 * q + 2] = acc[i][j][4 * q + 2] + bq[j][q].z;
        v[4 * q + 3] = acc[i][j][4 * q + 3] + bq[j][q].w;
      }
      if constexpr (KIND == EPI_GELU) {
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = gelu_erf(v[r]);
      }
      if constexpr (KIND == EPI_QKV) {
        // q columns (n < d, whole quads) carry the attention scale into exp2
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (n0w + j * 32 + 8 * q + 4 * lh < e.d_model)
#pragma unroll
            for (int r = 0; r < 4; ++r) v[4 * q + r] *= kQScaleLog2;
      }
      {
        uint32_t o[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          o[2 * q] = pack2_bf16(v[4 * q], v[4 * q + 1]);
          o[2 * q + 1] = pack2_bf16(v[4 * q + 2], v[4 * q + 3]);
        }
        // lanes 32-63 of quads 0 / 2 <-> lanes 0-31 of quads 1 / 3: lane l < 32
        // then holds columns 0-7 (16-23), lane l + 32 columns 8-15 (24-31)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const auto s0 = __builtin_amdgcn_permlane32_swap(o[4 * h], o[4 * h + 2], false, false);
          const auto s1 = __builtin_amdgcn_permlane32_swap(o[4 * h + 1], o[4 * h + 3], false, false);
          o[4 * h] = s0[0];
          o[4 * h + 2] = s0[1];
          o[4 * h + 1] = s1[0];
          o[4 * h + 3] = s1[1];
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int n = n0w + j * 32 + 16 * h + 8 * lh;
          const u32x4 x = {o[4 * h], o[4 * h + 1], o[4 * h + 2], o[4 * h + 3]};
          if constexpr (KIND == EPI_XKV) {
            if (rok && n < N)
              *(u32x4*)((bf16_t*)e.out + xrow[i] + xcol + (n - n0w)) = x;
          } else {
            const uint32_t off = rok && n < N ? (uint32_t)(rofs + n) * 2u : 0x80000000u;
            __builtin_amdgcn_raw_buffer_store_b128(x, rs, off, 0, kNtAux);
          }
        }
      }
    }
  }
}

template <int BM, int BN, int BK, int WM, int WN, int S, int KIND, bool SW>
__global__ __launch_bounds__(WM* WN * 64) __attribute__((amdgpu_waves_per_eu(2)))
void k_gemm_bf16_ps(AView a,
                                                             const bf16_t* __restrict__ w,
                                                             int M, int N, int K, Epilogue e,
                                                             int n_tm, int n_tn, int gm) {
  constexpr int NW = WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int CPR = BK / 8;
  constexpr int NS = BK / 16;
  constexpr int RPI = 1024 / (BK * 2);
  constexpr int IA = BM / (RPI * NW), IB = BN / (RPI * NW);
  constexpr int LPT = IA + IB;
  static_assert(BK == 32 || BK == 64, "BK");
  static_assert(NS % 2 == 0, "fragment double buffer parity");
  static_assert(IA * RPI * NW == BM && IB * RPI * NW == BN, "tile/waves");
  static_assert(S >= 2 && LPT * (S - 1) < 64, "stages");
  static_assert(FM + FN <= 15, "lgkmcnt");
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];
  constexpr int STAGE = (BM + BN) * BK;
  constexpr int kLgkmImm = 0xF | (0x3 << 14) | (0x7 << 4) | ((FM + FN) << 8);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WM, wn = wave / WM;
  const int n_tiles = n_tm * n_tn, grid = gridDim.x;
  if ((int)blockIdx.x >= n_tiles) return;
  const int my_tiles = (n_tiles - (int)blockIdx.x + grid - 1) / grid;
  const int nk = K / BK;
  const int total = my_tiles * nk;
  const uint32_t lds0 =
      (uint32_t)(uintptr_t)((__attribute__((address_space(3))) bf16_t*)smem);

  // per-wave LDS destinations (fixed) and per-lane source offsets in bytes
  // from a wave-uniform base (32-bit: the launcher checks the operand
  // extents), reset per tile
  uint32_t adst[IA], bdst[IB];
#pragma unroll
  for (int i = 0; i < IA; ++i)
    adst[i] = __builtin_amdgcn_readfirstlane(lds0 + (uint32_t)((i * NW + wave) * RPI * BK * 2));
#pragma unroll
  for (int i = 0; i < IB; ++i)
    bdst[i] = __builtin_amdgcn_readfirstlane(
        lds0 + (uint32_t)((BM * BK + (i * NW + wave) * RPI * BK) * 2));
  const bf16_t* abase = (const bf16_t*)a.ptr;
  uint32_t aoff[IA], boff[IB];
  int src_tile = -1;
  auto set_src = [&](int ti) {
    int tm, tn;
    tile_of((int)blockIdx.x + ti * grid, n_tiles, n_tm, n_tn, gm, tm, tn);
#pragma unroll
    for (int i = 0; i < IA; ++i) {
      const int row = (i * NW + wave) * RPI + lane / CPR;
      const int c = ((lane % CPR) ^ lds_swz<BK>(row)) * 8;
      const int r = min(tm * BM + row, M - 1);
      const int g = r / a.rows_per_batch;
      aoff[i] = (uint32_t)(g * a.batch_stride + (int64_t)(r - g * a.rows_per_batch) * a.lda + c) * 2u;
    }
#pragma unroll
    for (int i = 0; i < IB; ++i) {
      const int row = (i * NW + wave) * RPI + lane / CPR;
      const int c = ((lane % CPR) ^ lds_swz<BK>(row)) * 8;
      boff[i] = ((uint32_t)min(tn * BN + row, N - 1) * (uint32_t)K + (uint32_t)c) * 2u;
    }
    src_tile = ti;
  };
  auto issue = [&](int gi) {
    const int ti = gi / nk, kt = gi - ti * nk;
    if (ti != src_tile) set_src(ti);
    const uint32_t so = (uint32_t)((gi % S) * STAGE * 2);
    const bf16_t* ak = abase + kt * BK;
    const bf16_t* bk = w + kt * BK;
#pragma unroll
    for (int i = 0; i < IA; ++i) lds_dma16_s(adst[i] + so, aoff[i], ak);
#pragma unroll
    for (int i = 0; i < IB; ++i) lds_dma16_s(bdst[i] + so, boff[i], bk);
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int lrow = lane & 31, sw = lds_swz<BK>(lrow), lh = lane >> 5;
  const bf16_t* a_frag = smem + (wm * TM + lrow) * BK;
  const bf16_t* b_frag = smem + BM * BK + (wn * TN + lrow) * BK;
  bf16x8 af[2][FM], bfr[2][FN];
#define PS_READ(P, GI, KK)                                                            \
  do {                                                                                \
    const int off_ = ((GI) % S) * STAGE + ((((KK) * 2 + lh) ^ sw) * 8);               \
    _Pragma("unroll") for (int i = 0; i < FM; ++i)                                    \
      af[P][i] = *(const bf16x8*)(a_frag + off_ + i * 32 * BK);                       \
    _Pragma("unroll") for (int j = 0; j < FN; ++j)                                    \
      bfr[P][j] = *(const bf16x8*)(b_frag + off_ + j * 32 * BK);                      \
  } while (0)

#pragma unroll
  for (int t = 0; t < S; ++t)
    if (t < total) issue(t);
  wait_vm_lgkm0_rt<LPT*(S - 1)>(LPT * min(S - 1, total - 1));
  __builtin_amdgcn_s_barrier();
  PS_READ(0, 0, 0);
  // QKV: output tiles of V columns take the staged V^T epilogue, q / k tiles
  // the register one; 2 d_model is a multiple of the tile width, so a tile
  // never mixes them
  auto vt_of = [&](int t) {
    if constexpr (KIND != EPI_QKV) {
      return false;
    } else {
      int tm, tn;
      tile_of((int)blockIdx.x + t * grid, n_tiles, n_tm, n_tn, gm, tm, tn);
      return tn * BN >= 2 * e.d_model;
    }
  };
  bool tile_vt = vt_of(0);
  int ti = 0, kt = 0;
  for (int gi = 0; gi < total; ++gi) {
    const bool last_k = kt == nk - 1;
#pragma unroll
    for (int kk = 0; kk < NS; ++kk) {
      const int p = kk & 1;
      if (kk + 1 < NS) {
        PS_READ(p ^ 1, gi, kk + 1);
      } else if (!last_k) {
        wait_vm_lgkm0_rt<LPT*(S - 2)>(LPT * min(S - 2, total - 2 - gi));
        __builtin_amdgcn_s_barrier();
        if (gi + S < total) issue(gi + S);
        PS_READ(p ^ 1, gi + 1, 0);
      }
      if (kk + 1 < NS || !last_k) __builtin_amdgcn_s_waitcnt(kLgkmImm);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = SW ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[p][j], af[p][i], acc[i][j], 0, 0, 0)
                         : __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[p][i], bfr[p][j], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (last_k) {
      const bool more = gi + 1 < total;
      if (more) {
        // next K tile landed and every wave is done with this one
        wait_vm_lgkm0_rt<LPT*(S - 2)>(LPT * min(S - 2, total - 2 - gi));
        __builtin_amdgcn_s_barrier();
      }
      int tm, tn;
      tile_of((int)blockIdx.x + ti * grid, n_tiles, n_tm, n_tn, gm, tm, tn);
      if constexpr (SW && KIND == EPI_QKV) {
        if (tile_vt)
          epi_direct_vt<FM, FN>(e, acc, (float*)(smem + S * STAGE) + wave * 16 * kStageLd,
                                tm * BM + wm * TM, tn * BN + wn * TN, M, N, lane);
        else
          epi_direct<KIND, FM, FN>(e, acc, tm * BM + wm * TM, tn * BN + wn * TN, M, N, lane);
      } else if constexpr (SW)
        epi_direct<KIND, FM, FN>(e, acc, tm * BM + wm * TM, tn * BN + wn * TN, M, N, lane);
      else
        epi_wave_half<KIND, FM, FN>(e, acc, (float*)(smem + S * STAGE) + wave * 16 * kStageLd,
                                    tm * BM + wm * TM, tn * BN + wn * TN, M, N, lane);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
      if (more) {
        if (gi + S < total) issue(gi + S);
        PS_READ(0, gi + 1, 0);
      }
      ++ti;
      kt = 0;
      tile_vt = vt_of(ti);
    } else {
      ++kt;
    }
  }
#undef PS_READ
}

// CUs the persistent GEMM leaves free (0 by default); set while a prefill
// runs beside decode work on another stream, so that work finds CUs.
static int g_ps_reserve = 0;
void gemm_set_cu_reserve(int n) { g_ps_reserve = n < 0 ? 0 : n; }

template <int BM, int BN, int BK, int WM, int WN, int S, int KIND, int OCC = 1, bool SW = false>
static void launch_gemm_ps(const AView& a, const bf16_t* w, int M, int N, int K,
                           const Epilogue& e, hipStream_t s, int gm) {
  constexpr size_t lds = (size_t)S * (BM + BN) * BK * sizeof(bf16_t) +
                        (SW && KIND != EPI_QKV ? 0 : (size_t)WM * WN * 16 * kStageLd * sizeof(float));
  auto kfn = k_gemm_bf16_ps<BM, BN, BK, WM, WN, S, KIND, SW>;
  static bool attr = false;
  static int n_cu = 0;
  if (!attr) {
    (void)hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)lds);
    int dev = 0;
    (void)hipGetDevice(&dev);
    (void)hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
    if (n_cu <= 0) n_cu = 256;
    attr = true;
  }
  const int n_tm = (M + BM - 1) / BM, n_tn = (N + BN - 1) / BN;
  // keep the grid a multiple of 8 (one share per XCD) when CUs are reserved
  const int avail = g_ps_reserve > 0 ? std::max(8, (n_cu - g_ps_reserve) / 8 * 8) : n_cu;
  const int grid = std::min(n_tm * n_tn, OCC * avail);
  kfn<<<grid, WM * WN * 64, lds, s>>>(a, w, M, N, K, e, n_tm, n_tn, gm);
}

// The register epilogue stores 16-byte runs of eight columns through a
// buffer resource that spans the output (byte size below 2^31).
static bool direct_epi_ok(const Epilogue& e, int M, int N) {
  if (N % 8 != 0 || ((uintptr_t)e.out & 15) != 0) return false;
  if (e.kind == EPI_XKV) return e.d_model % 64 == 0 && e.slot_stride % 8 == 0;
  if (e.kind == EPI_QKV) {
    // tiles of 256 columns never mix q / k with V; V^T fits a buffer resource
    const int64_t vt_bytes = (int64_t)((M + kCtx - 1) / kCtx) * e.n_head * kHeadDim * kVtLd * 2;
    if (e.d_model % 128 != 0 || N != 3 * e.d_model || ((uintptr_t)e.out2 & 7) != 0 ||
        vt_bytes >= (int64_t)INT32_MAX)
      return false;
  }
  return e.ldc % 8 == 0 && e.ldc >= N && (int64_t)M * e.ldc * 2 < (int64_t)INT32_MAX;
}

// Operand extents that the persistent kernel's 32-bit byte offsets can
// address.
static bool fits_u32_offsets(const AView& a, int M, int N, int K) {
  const int64_t r = M - 1, g = r / a.rows_per_batch;
  const int64_t a_end = g * a.batch_stride + (r - g * a.rows_per_batch) * a.lda + K;
  return 2 * a_end < (int64_t)UINT32_MAX && 2 * (int64_t)N * K < (int64_t)UINT32_MAX;
}

template <int BM, int BN, int BK, int WM, int WN, int S, int KIND>
static void launch_gemm_pf(const AView& a, const bf16_t* w, int M, int N, int K,
                           const Epilogue& e, hipStream_t s, int gm) {
  constexpr size_t lds0 = (size_t)S * (BM + BN) * BK * sizeof(bf16_t);
  constexpr size_t lds_epi = (size_t)WM * WN * 32 * kStageLd * sizeof(float);
  constexpr size_t lds = lds0 > lds_epi ? lds0 : lds_epi;
  auto kfn = k_gemm_bf16_pf<BM, BN, BK, WM, WN, S, KIND>;
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)lds);
    attr = true;
  }
  int n_tm = (M + BM - 1) / BM, n_tn = (N + BN - 1) / BN;
  kfn<<<n_tm * n_tn, WM * WN * 64, lds, s>>>(a, w, M, N, K, e, n_tm, n_tn, gm);
}

template <int BM, int BN, int BK, int WM, int WN, int S, int KIND, int SCHED = 0>
static void launch_gemm_dma(const AView& a, const bf16_t* w, int M, int N, int K,
                            const Epilogue& e, hipStream_t s, int gm) {
  constexpr size_t lds0 = (size_t)S * (BM + BN) * BK * sizeof(bf16_t);
  constexpr size_t lds_epi = (size_t)WM * WN * 32 * kStageLd * sizeof(float);
  constexpr size_t lds = lds0 > lds_epi ? lds0 : lds_epi;
  auto kfn = k_gemm_bf16_dma<BM, BN, BK, WM, WN, S, KIND, SCHED>;
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)lds);
    attr = true;
  }
  int n_tm = (M + BM - 1) / BM, n_tn = (N + BN - 1) / BN;
  kfn<<<n_tm * n_tn, WM * WN * 64, lds, s>>>(a, w, M, N, K, e, n_tm, n_tn, gm);
}

template <int BM, int BN, int BK, int WM, int WN, int KIND>
static void launch_gemm_cfg(const AView& a, const bf16_t* w, int M, int N, int K,
                            const Epilogue& e, hipStream_t s, int gm) {
  constexpr size_t lds0 = (size_t)2 * (BM + BN) * BK * sizeof(bf16_t);
  constexpr size_t lds_epi = (size_t)WM * WN * 32 * kStageLd * sizeof(float);
  constexpr size_t lds = lds0 > lds_epi ? lds0 : lds_epi;
  auto kfn = k_gemm_bf16<BM, BN, BK, WM, WN, KIND>;
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)lds);
    attr = true;
  }
  int n_tm = (M + BM - 1) / BM, n_tn = (N + BN - 1) / BN;
  kfn<<<n_tm * n_tn, WM * WN * 64, lds, s>>>(a, w, M, N, K, e, n_tm, n_tn, gm);
}

// Tile choice by shape (measured on MI355X with the encoder's products):
// 256x256x64 tiles, two LDS stages, 8 waves of 128x64, fragment reads
// pipelined across K tiles, wherever K is a multiple of 64 and at least 512
// tiles exist -- persistent (epilogue overlapped with the next tile's loads)
// unless the epilogue reads the output (residual add); otherwise 256x128x32
// with three stages (8 waves of 64x64), and 128x128x32 with four stages when
// even those tiles would be too few to fill the chip.  K not a multiple of 32
// (the 80-mel first convolution) takes the register-path kernel, which
// zero-fills the K tail.
template <int KIND>
static void launch_gemm_bf16(const AView& a, const bf16_t* w, int M, int N, int K,
                             const Epilogue& e, hipStream_t s) {
  const long t256x128 = (long)((M + 255) / 256) * ((N + 127) / 128);
  const long t256x256 = (long)((M + 255) / 256) * ((N + 255) / 256);
  if (K % 32 != 0) {
    if (t256x128 >= 1024)
      launch_gemm_cfg<256, 128, 32, 4, 2, KIND>(a, w, M, N, K, e, s, 4);
    else
      launch_gemm_cfg<128, 128, 32, 2, 2, KIND>(a, w, M, N, K, e, s, 8);
  } else if (K % 64 == 0 && t256x256 >= 512) {
    // (the stem's scatter epilogue runs slower from the persistent kernel's
    // half-block stage than from the plain kernel's full-block one; the
    // fused QKV product goes persistent only with its register epilogue)
    if (KIND != EPI_CONV1 && fits_u32_offsets(a, M, N, K) &&
        (KIND != EPI_QKV || direct_epi_ok(e, M, N))) {
      const int gm = N >= 3072 ? 8 : 4;
      if constexpr (kDirectEpi<KIND>) {
        if (direct_epi_ok(e, M, N)) {
          launch_gemm_ps<256, 256, 64, 2, 4, 2, KIND, 1, true>(a, w, M, N, K, e, s, gm);
          return;
        }
      }
      launch_gemm_ps<256, 256, 64, 2, 4, 2, KIND>(a, w, M, N, K, e, s, gm);
    } else
      launch_gemm_pf<256, 256, 64, 2, 4, 2, KIND>(a, w, M, N, K, e, s, 4);
  } else if (t256x128 >= 512) {
    launch_gemm_pf<256, 128, 32, 4, 2, 3, KIND>(a, w, M, N, K, e, s, 4);
  } else {
    launch_gemm_dma<128, 128, 32, 2, 2, 4, KIND>(a, w, M, N, K, e, s, 8);
  }
}

void gemm_bf16(const AView& a, const bf16_t* w, int M, int N, int K, const Epilogue& e,
               hipStream_t s) {
  if (M <= 0 || N <= 0) return;
  switch (e.kind) {
    case EPI_STORE: launch_gemm_bf16<EPI_STORE>(a, w, M, N, K, e, s); break;
    case EPI_GELU: launch_gemm_bf16<EPI_GELU>(a, w, M, N, K, e, s); break;
    case EPI_CONV1: launch_gemm_bf16<EPI_CONV1>(a, w, M, N, K, e, s); break;
    case EPI_CONV2: launch_gemm_bf16<EPI_CONV2>(a, w, M, N, K, e, s); break;
    case EPI_XKV: launch_gemm_bf16<EPI_XKV>(a, w, M, N, K, e, s); break;
    case EPI_QKV: launch_gemm_bf16<EPI_QKV>(a, w, M, N, K, e, s); break;
  }
}

// ---------------------------------------------------------------------------
// fp32 GEMM (SIMT): 64x64 tile, 256 threads, 4x4 outputs per thread.
// ---------------------------------------------------------------------------
template <int KIND>
__global__ __launch_bounds__(256) void k_gemm_f32(AView a, const float* __restrict__ w, int M,
                                                  int N, int K, Epilogue e, int n_tn) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float As[BK][BM + 4];
  __shared__ float Bs[BK][BN + 4];
  const int tid = threadIdx.x;
  const int tn = blockIdx.x % n_tn, tm = blockIdx.x / n_tn;
  const int m0 = tm * BM, n0 = tn * BN;
  const int lr = tid >> 2, lk = (tid & 3) * 4;      // loader: row, k offset
  const int ar = m0 + lr, bn = n0 + lr;
  const float* ap = (const float*)a.ptr + arow_offset(a, ar < M ? ar : 0) + lk;
  const float* bp = w + (int64_t)(bn < N ? bn : 0) * K + lk;
  const int ty = tid >> 4, tx = tid & 15;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += BK) {
    float4 va = make_float4(0.f, 0.f, 0.f, 0.f), vb = va;
    if (ar < M && k0 + lk < K) va = *(const float4*)(ap + k0);
    if (bn < N && k0 + lk < K) vb = *(const float4*)(bp + k0);
    As[lk + 0][lr] = va.x; As[lk + 1][lr] = va.y; As[lk + 2][lr] = va.z; As[lk + 3][lr] = va.w;
    Bs[lk + 0][lr] = vb.x; Bs[lk + 1][lr] = vb.y; Bs[lk + 2][lr] = vb.z; Bs[lk + 3][lr] = vb.w;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < BK; ++k) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[k][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[k][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int row = m0 + ty * 4 + i, col = n0 + tx * 4 + j;
      if (row < M && col < N) epi_apply<KIND, float>(e, row, col, acc[i][j]);
    }
}

template <int KIND>
static void launch_gemm_f32(const AView& a, const float* w, int M, int N, int K,
                            const Epilogue& e, hipStream_t s) {
  int n_tm = (M + 63) / 64, n_tn = (N + 63) / 64;
  k_gemm_f32<KIND><<<n_tm * n_tn, 256, 0, s>>>(a, w, M, N, K, e, n_tn);
}

void gemm_f32(const AView& a, const float* w, int M, int N, int K, const Epilogue& e,
              hipStream_t s) {
  if (M <= 0 || N <= 0) return;
  switch (e.kind) {
    case EPI_STORE: launch_gemm_f32<EPI_STORE>(a, w, M, N, K, e, s); break;
    case EPI_GELU: launch_gemm_f32<EPI_GELU>(a, w, M, N, K, e, s); break;
    case EPI_CONV1: launch_gemm_f32<EPI_CONV1>(a, w, M, N, K, e, s); break;
    case EPI_CONV2: launch_gemm_f32<EPI_CONV2>(a, w, M, N, K, e, s); break;
    case EPI_XKV: launch_gemm_f32<EPI_XKV>(a, w, M, N, K, e, s); break;
  }
}

// ---------------------------------------------------------------------------
// Decode GEMMs and the vocabulary projection (skinny products)
// ---------------------------------------------------------------------------
// A decode step multiplies at most 128 rows by each weight matrix once, so
// the product streams the weights from HBM (128 flops per weight byte, far
// below the MFMA ridge) and the rows ride along from L2.  A block owns a
// strip of 32 WN weight rows (output columns) and all 128 row slots over a K
// range, in 64-deep chunks: each chunk's weight tile and activation tile go
// global -> LDS with global_load_lds_dwordx4, eight lanes per 128-byte row
// segment (whole cache lines per instruction), with the round-robin XOR
// swizzle of the encoder GEMM (16-byte slot c of row r holds chunk
// c ^ ((r >> 1) & 7): conflict-free fragment reads).  The two operands have
// rings of their own: the weights, which come cold from HBM, run NW chunks
// ahead (most of a block's strip is in flight at once); the activations, an
// L2 hit, run NX chunks ahead.  Wave w computes strip w % WN against 32 WN
// activation rows with v_mfma_f32_32x32x16_bf16: weight rows are the "A"
// operand, activation rows the "B" operand.
constexpr int SK_BK = 64;          // K per chunk

__device__ __forceinline__ int sk_swz(int row) { return (row >> 1) & 7; }

enum SkEpi : int32_t { SK_PARTIAL = 0, SK_BIAS = 1, SK_GELU = 2, SK_ARGMAX = 3 };

// Larger key = larger value, then lower index.  Any NaN gets the largest
// value key so that it always wins and the finishing pass reports it.
__device__ __forceinline__ uint64_t argmax_key(float v, int n) {
  uint32_t o = (v != v) ? 0xffffffffu : ordered_u32(v);
  return ((uint64_t)o << 32) | (uint64_t)(0xffffffffu - (uint32_t)n);
}

struct SkOut {
  void* out;            // PARTIAL: float [splits][D][N]; BIAS/GELU: bf16 [D][N]
  const float* bias;    // BIAS/GELU
  uint64_t* keys;       // ARGMAX: [D][N / 32] best key per 32-row tile
  float* logits;        // ARGMAX: optional float [D][N]
};

// Loads issued after chunk c's activation tile (which follows every earlier
// load in issue order): the prologue issues weight chunks 0 .. NW-2, then
// activation chunks 0 .. NX-2; iteration c' issues weight chunk c' + NW - 1,
// then activation chunk c' + NX - 1 (each only when it exists).
template <int NW, int NX>
__device__ __forceinline__ int sk_after(int c, int nck, int lpw, int lpx) {
  int n = 0;
  int first = c - NX + 2;                 // iterations that issued after X(c)
  if (c <= NX - 2) {
    n += lpx * max(0, min(NX - 2, nck - 1) - c);
    first = 0;
  }
  for (int i = first; i < c; ++i)
    n += (i + NW - 1 < nck ? lpw : 0) + (i + NX - 1 < nck ? lpx : 0);
  return n;
}

template <int WN, int NW, int NX, int EPI>
__global__ __launch_bounds__(256) void k_skinny_bf16(const bf16_t* __restrict__ x,
                                                     const bf16_t* __restrict__ w, int D, int N,
                                                     int K, int KC, SkOut o) {
  constexpr int RB = WN;                         // row blocks of 32 per wave
  constexpr int WR = 32 * WN;                    // weight rows per block
  constexpr int WSTAGE = WR * SK_BK, XSTAGE = 128 * SK_BK;   // elements per ring stage
  constexpr int LPW = WN, LPX = 4;               // DMA instructions per wave per chunk
  constexpr int MAXOUT = (NW - 1) * LPW + (NX - 1) * LPX;
  static_assert(MAXOUT < 64, "vmcnt");
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];
  bf16_t* wring = smem;
  bf16_t* xring = smem + NW * WSTAGE;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l32 = lane & 31, lh = lane >> 5;
  const int n0 = blockIdx.x * WR, split = blockIdx.y;
  const int kb = split * KC, nck = KC / SK_BK;
  const uint32_t lds0 = (uint32_t)(uintptr_t)((__attribute__((address_space(3))) bf16_t*)smem);
  const uint32_t xlds0 = lds0 + (uint32_t)(NW * WSTAGE * 2);
  // DMA: instruction i of a wave fills rows 8 i .. 8 i + 7 of its share; lane
  // l lands at slot l % 8 of row l / 8 and fetches chunk (l % 8) ^ swz(row)
  uint32_t xdst[4], wdst[WN], xoff[4], woff[WN];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = wave * 32 + i * 8;                               // activation rows
    xdst[i] = __builtin_amdgcn_readfirstlane(xlds0 + (uint32_t)(row * SK_BK * 2));
    const int r = row + (lane >> 3);
    xoff[i] = (uint32_t)(((int64_t)min(r, D - 1) * K + kb + (((lane & 7) ^ sk_swz(r)) * 8)) * 2);
  }
#pragma unroll
  for (int i = 0; i < WN; ++i) {
    const int row = wave * 8 * WN + i * 8;                           // weight rows
    wdst[i] = __builtin_amdgcn_readfirstlane(lds0 + (uint32_t)(row * SK_BK * 2));
    const int r = row + (lane >> 3);
    woff[i] = (uint32_t)(((int64_t)min(n0 + r, N - 1) * K + kb + (((lane & 7) ^ sk_swz(r)) * 8)) * 2);
  }
  auto issue_w = [&](int c) {
    const uint32_t so = (uint32_t)((c % NW) * WSTAGE * 2);
    const bf16_t* wk = w + c * SK_BK;
#pragma unroll
    for (int i = 0; i < WN; ++i) lds_dma16_s(wdst[i] + so, woff[i], wk);
  };
  auto issue_x = [&](int c) {
    const uint32_t so = (uint32_t)((c % NX) * XSTAGE * 2);
    const bf16_t* xk = x + c * SK_BK;
#pragma unroll
    for (int i = 0; i < 4; ++i) lds_dma16_s(xdst[i] + so, xoff[i], xk);
  };
  const int strip = wave % WN, rg = wave / WN;                      // this wave's strip, row group
  const int wrow = strip * 32 + l32, sww = sk_swz(wrow);
  int xrow[RB], swx[RB];
#pragma unroll
  for (int j = 0; j < RB; ++j) {
    xrow[j] = (rg * RB + j) * 32 + l32;
    swx[j] = sk_swz(xrow[j]);
  }
  f32x16 acc[RB];
#pragma unroll
  for (int j = 0; j < RB; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;

  for (int c = 0; c < NW - 1 && c < nck; ++c) issue_w(c);
  for (int c = 0; c < NX - 1 && c < nck; ++c) issue_x(c);
  for (int c = 0; c < nck; ++c) {
    // this wave's tiles of chunk c have landed once at most the loads issued
    // after them are outstanding; the barrier then publishes every wave's
    // share and frees the stages of chunk c - 1 for the next issues
    wait_vmcnt_rt<MAXOUT>(sk_after<NW, NX>(c, nck, LPW, LPX));
    __builtin_amdgcn_s_barrier();
    if (c + NW - 1 < nck) issue_w(c + NW - 1);
    if (c + NX - 1 < nck) issue_x(c + NX - 1);
    const bf16_t* wt = wring + (c % NW) * WSTAGE;
    const bf16_t* xt = xring + (c % NX) * XSTAGE;
    bf16x8 wf[4], xf[4][RB];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int ch = kk * 2 + lh;
      wf[kk] = *(const bf16x8*)(wt + wrow * SK_BK + ((ch ^ sww) * 8));
#pragma unroll
      for (int j = 0; j < RB; ++j)
        xf[kk][j] = *(const bf16x8*)(xt + xrow[j] * SK_BK + ((ch ^ swx[j]) * 8));
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int j = 0; j < RB; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[kk], xf[kk][j], acc[j], 0, 0, 0);
  }
  // lane holds activation row xrow[j] and weight rows (output columns)
  // n0 + strip 32 + 8 (r / 4) + 4 (lane / 32) + r % 4
  const int nb = n0 + strip * 32;
#pragma unroll
  for (int j = 0; j < RB; ++j) {
    const int row = xrow[j];
    if constexpr (EPI == SK_ARGMAX) {
      uint64_t best = 0;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int n = nb + (r >> 2) * 8 + lh * 4 + (r & 3);
        if (n < N) {
          const uint64_t kk = argmax_key(acc[j][r], n);
          best = kk > best ? kk : best;
          if (o.logits && row < D) o.logits[(int64_t)row * N + n] = acc[j][r];
        }
      }
      const uint32_t plo = __shfl_xor((uint32_t)best, 32, 64);
      const uint32_t phi = __shfl_xor((uint32_t)(best >> 32), 32, 64);
      const uint64_t other = ((uint64_t)phi << 32) | plo;
      best = other > best ? other : best;
      const int n_tiles = (N + 31) / 32;
      if (lane < 32 && row < D && nb < N) o.keys[(int64_t)row * n_tiles + nb / 32] = best;
    } else {
      if (row >= D) continue;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = nb + g * 8 + lh * 4;
        float4 v = make_float4(acc[j][g * 4], acc[j][g * 4 + 1], acc[j][g * 4 + 2],
                               acc[j][g * 4 + 3]);
        if constexpr (EPI == SK_PARTIAL) {
          *(float4*)((float*)o.out + ((int64_t)split * D + row) * N + n) = v;
        } else {
          v = add4(v, *(const float4*)(o.bias + n));
          if constexpr (EPI == SK_GELU) v = gelu4(v);
          typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
          u32x2 u;
          u.x = pack2_bf16(v.x, v.y);
          u.y = pack2_bf16(v.z, v.w);
          *(u32x2*)((bf16_t*)o.out + (int64_t)row * N + n) = u;
        }
      }
    }
  }
}

template <int WN, int NW, int NX, int EPI>
static void launch_skinny(const bf16_t* x, const bf16_t* w, int D, int N, int K, int splits,
                          const SkOut& o, hipStream_t s) {
  constexpr size_t lds = ((size_t)NW * 32 * WN + (size_t)NX * 128) * SK_BK * sizeof(bf16_t);
  static_assert(lds <= 160 * 1024, "LDS");
  auto kfn = k_skinny_bf16<WN, NW, NX, EPI>;
  static bool attr = false;
  if (!attr) {
    (void)hipFuncSetAttribute((const void*)kfn, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)lds);
    attr = true;
  }
  dim3 grid((N + 32 * WN - 1) / (32 * WN), splits);
  kfn<<<grid, 256, lds, s>>>(x, w, D, N, K, K / splits, o);
}

// K slices of a partial-sum product: the largest divisor of K / 64 that keeps
// the grid (N / 32 strips x slices) within one block per CU, at most 16.
int dgemm_splits(int N, int K) {
  const int tiles = N / 32, q = K / 64;
  int best = 1;
  for (int sp = 1; sp <= 16 && sp <= q; ++sp)
    if (q % sp == 0 && tiles * sp <= 256) best = sp;
  return best;
}

int dgemm_bf16(const bf16_t* x, const bf16_t* w, int D, int N, int K, int epi,
               const float* bias, void* out, hipStream_t s) {
  // N % 32 == 0, K % 64 == 0 and D <= 128 are checked when the context is created
  if (D <= 0) return 1;
  SkOut o{out, bias, nullptr, nullptr};
  // weight ring 16 x 4 KB (15 chunks in flight), activation ring 3 x 16 KB
  if (epi == DG_PARTIAL) {
    const int sp = dgemm_splits(N, K);
    launch_skinny<1, 16, 3, SK_PARTIAL>(x, w, D, N, K, sp, o, s);
    return sp;
  }
  if (epi == DG_GELU)
    launch_skinny<1, 16, 3, SK_GELU>(x, w, D, N, K, 1, o, s);
  else
    launch_skinny<1, 16, 3, SK_BIAS>(x, w, D, N, K, 1, o, s);
  return 1;
}

void dgemm_f32(const float* x, const float* w, int D, int N, int K, float* out, hipStream_t s) {
  AView a{x, K, 0, 1 << 30};
  Epilogue e{};
  e.kind = EPI_STORE;
  e.out = out;
  e.ldc = N;
  gemm_f32(a, w, D, N, K, e, s);
}

template <typename T>
__global__ void k_dgemm_reduce(const float* partial, int splits, int D, int N,
                               const float* bias, int mode, void* out) {
  int64_t n_all = (int64_t)D * N;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n_all;
       i += (int64_t)gridDim.x * blockDim.x) {
    int n = (int)(i % N);
    float v = bias ? bias[n] : 0.f;
    for (int s = 0; s < splits; ++s) v += partial[(int64_t)s * n_all + i];
    if (mode == 0) {
      St<T>::st((T*)out, i, v);
    } else if (mode == 1) {
      St<T>::st((T*)out, i, gelu_erf(v));
    } else {
      ((float*)out)[i] += v;
    }
  }
}
template <typename T>
void dgemm_reduce(const float* partial, int splits, int D, int N, const float* bias, int mode,
                  void* out, hipStream_t s) {
  int64_t n = (int64_t)D * N;
  if (n <= 0) return;
  int g = (int)((n + 255) / 256);
  if (g > 8192) g = 8192;
  k_dgemm_reduce<T><<<g, 256, 0, s>>>(partial, splits, D, N, bias, mode, out);
}
template void dgemm_reduce<float>(const float*, int, int, int, const float*, int, void*,
                                  hipStream_t);
template void dgemm_reduce<bf16_t>(const float*, int, int, int, const float*, int, void*,
                                   hipStream_t);

// Split-K reduce fused with the residual add and the next LayerNorm: one
// block per decode row.  Thread t sums the float4 column group t % G (G =
// d/4) over the splits s = t / G, t / G + SG, ... (SG split groups, unrolled
// so that several loads are in flight), the SG partial sums meet in LDS, and
// the G owners finish the row:  h[b] += bias + sum_s partial[s][b];
// xn[b] = LN(h[b]) (eps 1e-5).
template <typename T>
__global__ __launch_bounds__(1024) void k_reduce_resid_ln(const float* __restrict__ partial,
                                                          int splits, int D, int d,
                                                          const float* __restrict__ bias,
                                                          float* __restrict__ h,
                                                          const float* __restrict__ g,
                                                          const float* __restrict__ beta, T* xn) {
  __shared__ float4 part[1024];
  __shared__ float red[2][16];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int G = d >> 2, SG = blockDim.x / G;
  const int grp = tid % G, sg = tid / G;
  const int64_t rs = (int64_t)D * d;                 // stride between splits
  const float* src = partial + (int64_t)b * d + grp * 4;
  // the owners' row, bias and LayerNorm parameters load beside the partials
  // (one memory round trip for the whole kernel)
  float4 hv = make_float4(0.f, 0.f, 0.f, 0.f), bv = hv, gg = hv, bb = hv;
  float* hp = h + (int64_t)b * d + tid * 4;
  if (tid < G) {
    hv = *(const float4*)hp;
    bv = *(const float4*)(bias + tid * 4);
    gg = *(const float4*)(g + tid * 4);
    bb = *(const float4*)(beta + tid * 4);
  }
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
  if (sg < SG) {
    int s = sg;
    for (; s + 3 * SG < splits; s += 4 * SG) {
      const float4 v0 = *(const float4*)(src + s * rs);
      const float4 v1 = *(const float4*)(src + (s + SG) * rs);
      const float4 v2 = *(const float4*)(src + (s + 2 * SG) * rs);
      const float4 v3 = *(const float4*)(src + (s + 3 * SG) * rs);
      a = add4(a, add4(add4(v0, v1), add4(v2, v3)));
    }
    for (; s < splits; s += SG) a = add4(a, *(const float4*)(src + s * rs));
  }
  part[tid] = a;
  __syncthreads();
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  float sum = 0.f;
  if (tid < G) {
    for (int k = 1; k < SG; ++k) a = add4(a, part[tid + k * G]);
    v = add4(add4(hv, bv), a);
    *(float4*)hp = v;
    sum = (v.x + v.y) + (v.z + v.w);
  }
  const int nw = (blockDim.x + 63) >> 6;
  sum = wave_sum(sum);
  if (lane == 0) red[0][wave] = sum;
  __syncthreads();
  float tot = 0.f;
  for (int w2 = 0; w2 < nw; ++w2) tot += red[0][w2];
  const float mean = tot / d;
  float q = 0.f;
  if (tid < G) {
    const float4 c = make_float4(v.x - mean, v.y - mean, v.z - mean, v.w - mean);
    q = (c.x * c.x + c.y * c.y) + (c.z * c.z + c.w * c.w);
  }
  q = wave_sum(q);
  if (lane == 0) red[1][wave] = q;
  __syncthreads();
  float var = 0.f;
  for (int w2 = 0; w2 < nw; ++w2) var += red[1][w2];
  const float rstd = rsqrtf(var / d + 1e-5f);
  if (tid < G) {
    const float o[4] = {(v.x - mean) * rstd * gg.x + bb.x, (v.y - mean) * rstd * gg.y + bb.y,
                        (v.z - mean) * rstd * gg.z + bb.z, (v.w - mean) * rstd * gg.w + bb.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) St<T>::st(xn, (int64_t)b * d + tid * 4 + k, o[k]);
  }
}

template <typename T>
void reduce_resid_ln(const float* partial, int splits, int D, int d, const float* bias, float* h,
                     const float* g, const float* beta, T* xn, hipStream_t s) {
  if (D <= 0) return;
  const int G = d / 4;                                // d % 64 == 0, d <= 2048
  const int SG = std::max(1, 1024 / G);
  const int threads = (G * SG + 63) / 64 * 64;
  k_reduce_resid_ln<T><<<D, threads, 0, s>>>(partial, splits, D, d, bias, h, g, beta, xn);
}
template void reduce_resid_ln<float>(const float*, int, int, int, const float*, float*,
                                     const float*, const float*, float*, hipStream_t);
template void reduce_resid_ln<bf16_t>(const float*, int, int, int, const float*, float*,
                                      const float*, const float*, bf16_t*, hipStream_t);

// ---------------------------------------------------------------------------
// Vocabulary projection + argmax
// ---------------------------------------------------------------------------
int vocab_tiles(int V) { return (V + 31) / 32; }

// The vocabulary projection is the skinny product with 128 vocabulary rows per
// block (each wave one 32-row strip against all 128 row slots, so the
// activations are read once per 128 vocabulary rows); each wave leaves, for
// each decode row, the best key over its 32-row vocabulary tile.
void vocab_argmax_bf16(const bf16_t* x, const bf16_t* emb, int D, int V, int K, uint64_t* keys,
                       int n_tiles, float* logits, hipStream_t s) {
  if (D <= 0) return;
  (void)n_tiles;   // = vocab_tiles(V): the kernel derives it from V
  SkOut o{nullptr, nullptr, keys, logits};
  // 128 vocabulary rows per block with a 3-chunk weight and 2-chunk
  // activation ring (80 KB of LDS): two blocks per CU, so the 406 blocks of
  // the 51866-row table are all resident at once instead of running in a
  // full round and a partial one
  launch_skinny<4, 3, 2, SK_ARGMAX>(x, emb, D, V, K, 1, o, s);
}

void vocab_logits_f32(const float* x, const float* emb, int D, int V, int K, float* logits,
                      hipStream_t s) {
  AView a{x, K, 0, 1 << 30};
  Epilogue e{};
  e.kind = EPI_STORE;
  e.out = logits;
  e.ldc = V;
  gemm_f32(a, emb, D, V, K, e, s);
}

__global__ void k_logits_keys(const float* logits, int D, int V, uint64_t* keys, int n_tiles) {
  int tile = blockIdx.x, b = blockIdx.y;
  int n = tile * 32 + threadIdx.x;                 // 32-entry tiles, upper lanes idle
  uint64_t best = 0;
  if (threadIdx.x < 32 && n < V) best = argmax_key(logits[(int64_t)b * V + n], n);
  for (int o = 32; o > 0; o >>= 1) {
    uint32_t lo = __shfl_xor((uint32_t)best, o, 64), hi = __shfl_xor((uint32_t)(best >> 32), o, 64);
    uint64_t other = ((uint64_t)hi << 32) | lo;
    best = other > best ? other : best;
  }
  if (threadIdx.x == 0) keys[(int64_t)b * n_tiles + tile] = best;
}
void logits_argmax_keys(const float* logits, int D, int V, uint64_t* keys, int n_tiles,
                        hipStream_t s) {
  if (D > 0) k_logits_keys<<<dim3(n_tiles, D), 64, 0, s>>>(logits, D, V, keys, n_tiles);
}

// One wave per row: max key over the row's tiles; NaN winner raises the flag.
__global__ void k_argmax_finish(const uint64_t* keys, int n_tiles, int32_t* out,
                                int32_t* nan_flag) {
  int b = blockIdx.x;
  uint64_t best = 0;
  for (int t = threadIdx.x; t < n_tiles; t += 64) {
    uint64_t k = keys[(int64_t)b * n_tiles + t];
    best = k > best ? k : best;
  }
  for (int o = 32; o > 0; o >>= 1) {
    uint32_t lo = __shfl_xor((uint32_t)best, o, 64), hi = __shfl_xor((uint32_t)(best >> 32), o, 64);
    uint64_t other = ((uint64_t)hi << 32) | lo;
    best = other > best ? other : best;
  }
  if (threadIdx.x == 0) {
    float v = from_ordered_u32((uint32_t)(best >> 32));
    out[b] = (int32_t)(0xffffffffu - (uint32_t)best);
    if (v != v) atomicOr(nan_flag, 1);
  }
}
void argmax_finish(const uint64_t* keys, int D, int n_tiles, int32_t* out, int32_t* nan_flag,
                   hipStream_t s) {
  if (D > 0) k_argmax_finish<<<D, 64, 0, s>>>(keys, n_tiles, out, nan_flag);
}

}  // namespace asr
