// GEMMs of the step.
//
//  * gemm_bf16: C = A . W^T on gfx950 MFMA (v_mfma_f32_32x32x16_bf16), bf16
//    operands, fp32 accumulation, LDS double buffering, fused epilogues
//    (bias, exact GELU, fp32 residual add, conv-stem row mapping, scatter of
//    all decoder layers' cross K/V into a slot's cache).
//  * gemm_f32: the same contract in plain fp32 FMA (the fp32 model path).
//  * dgemm_bf16 / dgemm_f32: skinny products for the decode rows with K split
//    across workgroups (weights streamed once), then a reduce kernel that
//    applies the epilogue.
//  * vocab_argmax_bf16: the tied vocabulary projection fused with a per-row
//    argmax (lowest index on ties) over each 64-column tile, finished by a
//    deterministic cross-tile reduction.
#include "asr_device.h"

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
  } else if constexpr (KIND == EPI_RESID) {
    float* x = (float*)e.out + (int64_t)r * e.ldc + n;
    *x = *x + v;
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
      St<T>::st((T*)e.out, (int64_t)r * e.ldc + n, v);
    } else {
      int g = r / kCtx, t = r - g * kCtx;
      int hd = n - two_d;
      int64_t addr = (((int64_t)g * e.n_head + (hd >> 6)) * kHeadDim + (hd & 63)) * kVtLd + t;
      St<T>::st((T*)e.out2, addr, v);
    }
  }
}

// Epilogue of one 32x32 accumulator block staged in LDS (row stride 33).  V
// blocks of the fused QKV product are walked column-major so that lanes run
// along positions, the contiguous direction of the transposed V.
template <int KIND>
__device__ __forceinline__ void epi_block(const Epilogue& e, const float* stage, int rbase,
                                          int cbase, int M, int N, int lane) {
  const int l32 = lane & 31, lh = lane >> 5;
  if (KIND == EPI_QKV && cbase >= 2 * e.d_model) {
#pragma unroll 2
    for (int t = 0; t < 16; ++t) {
      const int cc = t * 2 + lh;
      const int row = rbase + l32, col = cbase + cc;
      if (row < M && col < N) epi_apply<KIND, bf16_t>(e, row, col, stage[l32 * 33 + cc]);
    }
  } else {
#pragma unroll 2
    for (int t = 0; t < 16; ++t) {
      const int rr = t * 2 + lh;
      const int row = rbase + rr, col = cbase + l32;
      if (row < M && col < N) epi_apply<KIND, bf16_t>(e, row, col, stage[rr * 33 + l32]);
    }
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
#ifndef ASR_GEMM_CEILING_PROBE
    if (kt + 1 < nk) GEMM_GLOAD(ra, rb, (kt + 1) * BK);
#endif
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
#ifndef ASR_GEMM_CEILING_PROBE
    if (kt + 1 < nk) GEMM_SSTORE(ra, rb, cur ^ 1);
#endif
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
  float* stage = (float*)smem + wave * (32 * 33);
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        stage[((r >> 2) * 8 + (lane >> 5) * 4 + (r & 3)) * 33 + lrow] = acc[i][j][r];
      __syncthreads();
      epi_block<KIND>(e, stage, m0 + wm * TM + i * 32, n0 + wn * TN + j * 32, M, N, lane);
      __syncthreads();
    }
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

template <int BM, int BN, int BK, int WM, int WN, int S, int KIND>
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
    }
  }
  wait_vmcnt<0>();
  __syncthreads();

  float* stage = (float*)smem + wave * (32 * 33);
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        stage[((r >> 2) * 8 + (lane >> 5) * 4 + (r & 3)) * 33 + lrow] = acc[i][j][r];
      __syncthreads();
      epi_block<KIND>(e, stage, m0 + wm * TM + i * 32, n0 + wn * TN + j * 32, M, N, lane);
      __syncthreads();
    }
}

template <int BM, int BN, int BK, int WM, int WN, int S, int KIND>
static void launch_gemm_dma(const AView& a, const bf16_t* w, int M, int N, int K,
                            const Epilogue& e, hipStream_t s, int gm) {
  constexpr size_t lds0 = (size_t)S * (BM + BN) * BK * sizeof(bf16_t);
  constexpr size_t lds_epi = (size_t)WM * WN * 32 * 33 * sizeof(float);
  constexpr size_t lds = lds0 > lds_epi ? lds0 : lds_epi;
  auto kfn = k_gemm_bf16_dma<BM, BN, BK, WM, WN, S, KIND>;
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
  constexpr size_t lds_epi = (size_t)WM * WN * 32 * 33 * sizeof(float);
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
// deep-K products (K >= 2048) use 256x256x64 tiles, two LDS stages, 8 waves of
// 128x64; the rest 256x128x32 with three stages, 8 waves of 64x64; small
// products 128x128x32 with four stages so that enough workgroups exist.  K not
// a multiple of 32 (the 80-mel first convolution) takes the register-path
// kernel, which zero-fills the K tail.
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
  } else if (K >= 2048 && K % 64 == 0 && t256x256 >= 512) {
    launch_gemm_dma<256, 256, 64, 2, 4, 2, KIND>(a, w, M, N, K, e, s, 4);
  } else if (t256x128 >= 512) {
    launch_gemm_dma<256, 128, 32, 4, 2, 3, KIND>(a, w, M, N, K, e, s, 4);
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
    case EPI_RESID: launch_gemm_bf16<EPI_RESID>(a, w, M, N, K, e, s); break;
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
    case EPI_RESID: launch_gemm_f32<EPI_RESID>(a, w, M, N, K, e, s); break;
    case EPI_CONV1: launch_gemm_f32<EPI_CONV1>(a, w, M, N, K, e, s); break;
    case EPI_CONV2: launch_gemm_f32<EPI_CONV2>(a, w, M, N, K, e, s); break;
    case EPI_XKV: launch_gemm_f32<EPI_XKV>(a, w, M, N, K, e, s); break;
  }
}

// ---------------------------------------------------------------------------
// Decode GEMMs
// ---------------------------------------------------------------------------
// One block: 64 output columns x all decode rows (one wave per 32 rows) over
// one K-split.  The weight rows are the MFMA "A" operand, the activation rows
// the "B" operand, so each lane ends with one row's values for 16 columns.
__global__ __launch_bounds__(256) void k_dgemm_bf16(const bf16_t* __restrict__ x,
                                                    const bf16_t* __restrict__ w, int D, int N,
                                                    int K, int kc, float* partial) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * 64, split = blockIdx.y;
  const int kb = split * kc, ke = min(K, kb + kc);
  const int b0 = wave * 32;
  if (b0 >= D) return;
  const int brow = b0 + (lane & 31);
  const int lk = (lane >> 5) * 8;
  const bf16_t* xp = x + (int64_t)min(brow, D - 1) * K + lk;
  const bf16_t* wp0 = w + (int64_t)min(n0 + (lane & 31), N - 1) * K + lk;
  const bf16_t* wp1 = w + (int64_t)min(n0 + 32 + (lane & 31), N - 1) * K + lk;
  f32x16 acc0, acc1;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc0[r] = acc1[r] = 0.f;
#pragma unroll 4
  for (int k = kb; k < ke; k += 16) {
    bf16x8 xb = *(const bf16x8*)(xp + k);
    bf16x8 w0 = *(const bf16x8*)(wp0 + k);
    bf16x8 w1 = *(const bf16x8*)(wp1 + k);
    acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(w0, xb, acc0, 0, 0, 0);
    acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(w1, xb, acc1, 0, 0, 0);
  }
  if (brow >= D) return;
  float* out = partial + ((int64_t)split * D + brow) * N;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    int n = n0 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
    if (n < N) out[n] = acc0[r];
    if (n + 32 < N) out[n + 32] = acc1[r];
  }
}

static int choose_kc(int N, int K, int max_splits) {
  // aim for >= ~512 workgroups while keeping each split >= 128 deep
  int n_tiles = (N + 63) / 64;
  int splits = (512 + n_tiles - 1) / n_tiles;
  int max_by_depth = K / 128 > 0 ? K / 128 : 1;
  if (splits > max_by_depth) splits = max_by_depth;
  if (splits > max_splits) splits = max_splits;
  if (splits < 1) splits = 1;
  int kc = (K + splits - 1) / splits;
  kc = (kc + 15) / 16 * 16;
  return kc;
}

int dgemm_bf16(const bf16_t* x, const bf16_t* w, int D, int N, int K, float* partial,
               int max_splits, hipStream_t s) {
  int kc = choose_kc(N, K, max_splits);
  int splits = (K + kc - 1) / kc;
  dim3 grid((N + 63) / 64, splits);
  if (D > 0) k_dgemm_bf16<<<grid, 256, 0, s>>>(x, w, D, N, K, kc, partial);
  return splits;
}

int dgemm_f32(const float* x, const float* w, int D, int N, int K, float* partial,
              int max_splits, hipStream_t s) {
  (void)max_splits;
  AView a{x, K, 0, 1 << 30};
  Epilogue e{};
  e.kind = EPI_STORE;
  e.out = partial;
  e.ldc = N;
  gemm_f32(a, w, D, N, K, e, s);
  return 1;
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

// ---------------------------------------------------------------------------
// Vocabulary projection + argmax
// ---------------------------------------------------------------------------
int vocab_tiles(int V) { return (V + 63) / 64; }

// Larger key = larger value, then lower index.  Any NaN gets the largest
// value key so that it always wins and the finishing pass reports it.
__device__ __forceinline__ uint64_t argmax_key(float v, int n) {
  uint32_t o = (v != v) ? 0xffffffffu : ordered_u32(v);
  return ((uint64_t)o << 32) | (uint64_t)(0xffffffffu - (uint32_t)n);
}

__global__ __launch_bounds__(256) void k_vocab_bf16(const bf16_t* __restrict__ x,
                                                    const bf16_t* __restrict__ emb, int D, int V,
                                                    int K, uint64_t* keys, int n_tiles,
                                                    float* logits) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * 64;
  const int b0 = wave * 32;
  if (b0 >= D) return;
  const int brow = b0 + (lane & 31);
  const int lk = (lane >> 5) * 8;
  const bf16_t* xp = x + (int64_t)min(brow, D - 1) * K + lk;
  const bf16_t* wp0 = emb + (int64_t)min(n0 + (lane & 31), V - 1) * K + lk;
  const bf16_t* wp1 = emb + (int64_t)min(n0 + 32 + (lane & 31), V - 1) * K + lk;
  f32x16 acc0, acc1;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc0[r] = acc1[r] = 0.f;
#pragma unroll 4
  for (int k = 0; k < K; k += 16) {
    bf16x8 xb = *(const bf16x8*)(xp + k);
    bf16x8 w0 = *(const bf16x8*)(wp0 + k);
    bf16x8 w1 = *(const bf16x8*)(wp1 + k);
    acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(w0, xb, acc0, 0, 0, 0);
    acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(w1, xb, acc1, 0, 0, 0);
  }
  uint64_t best = 0;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    int n = n0 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
    if (n < V) {
      uint64_t k0 = argmax_key(acc0[r], n);
      best = k0 > best ? k0 : best;
      if (logits && brow < D) logits[(int64_t)brow * V + n] = acc0[r];
    }
    if (n + 32 < V) {
      uint64_t k1 = argmax_key(acc1[r], n + 32);
      best = k1 > best ? k1 : best;
      if (logits && brow < D) logits[(int64_t)brow * V + n + 32] = acc1[r];
    }
  }
  uint32_t lo = (uint32_t)best, hi = (uint32_t)(best >> 32);
  uint32_t plo = __shfl_xor(lo, 32, 64), phi = __shfl_xor(hi, 32, 64);
  uint64_t other = ((uint64_t)phi << 32) | plo;
  best = other > best ? other : best;
  if (lane < 32 && brow < D) keys[(int64_t)brow * n_tiles + blockIdx.x] = best;
}

void vocab_argmax_bf16(const bf16_t* x, const bf16_t* emb, int D, int V, int K, uint64_t* keys,
                       int n_tiles, float* logits, hipStream_t s) {
  if (D > 0) k_vocab_bf16<<<n_tiles, 256, 0, s>>>(x, emb, D, V, K, keys, n_tiles, logits);
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
  int n = tile * 64 + threadIdx.x;
  uint64_t best = 0;
  if (n < V) best = argmax_key(logits[(int64_t)b * V + n], n);
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
