// Attention kernels.
//
//  * flash_attn_bf16: encoder self-attention over the 1500 positions of a
//    30-s segment (no mask), MFMA-based.  Each wave owns 32 queries; K and
//    V^T tiles of 64 keys are staged in LDS and shared by the block's
//    waves.  The kernel computes S^T = K Q^T so that, in the MFMA output
//    layout, each lane holds one query's scores for 32 keys: the row max
//    needs a single cross-lane exchange, the probabilities feed the
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

// ---------------------------------------------------------------------------
// Encoder flash attention (bf16)
//
// Block = 8 waves x 32 queries of one (clip, head); tiles of 64 keys.  K
// comes from the fused QKV buffer, V from the per-head transposed copy the
// QKV GEMM writes (V^T[dim][position], zero past 1500).  S^T = K Q^T is
// computed per 32-key x 32-query block, so in the MFMA output layout a lane
// owns one query: the row max needs one cross-lane exchange (lane ^ 32) and
// the online-softmax rescale is per lane.
//  * The K rows of each 32-key block enter the MFMA in the order that swaps
//    bits 2 and 3 of the row index.  A lane then holds its query's scores
//    for 8 consecutive keys per 16-key group, which, packed to bf16, are
//    directly the B operand of O^T += V^T P^T; the matching A operand is one
//    16-byte chunk of a V^T row.  Both tiles are plain [row][64] bf16 tiles
//    with 16-byte chunks XOR-swizzled by (row / 2) % 8 (conflict-free
//    fragment reads), double-buffered in LDS and filled by direct
//    global-to-LDS loads (one 1 KB instruction per wave per operand): tile
//    kt+1 is in flight while tile kt is consumed, one barrier per tile.
//  * The probability sum uses v_dot2 on the packed bf16 probabilities (the
//    same rounded values the P V product uses), two per instruction.
//  * Q arrives scaled by 1/sqrt(64) log2(e) (the QKV epilogue folds the
//    factor in before its one bf16 rounding), so scores are in the exp2
//    domain; softmax in fp32 with exp2 and a lazy reference (below).
// The kernel keeps to 128 VGPRs (four waves per SIMD, two blocks per CU):
// the exp2 work on the VALU and the MFMAs of other waves then overlap.
// ---------------------------------------------------------------------------
constexpr int FP_NW = 8, FP_KT = 64;

__device__ __forceinline__ void fp_dma16(uint32_t lds_addr, uint32_t voff, const void* sbase) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
               :: "s"(lds_addr), "v"(voff), "s"(sbase) : "memory", "m0");
}
template <int N>
__device__ __forceinline__ void fp_wait_vmcnt() {
  static_assert(N >= 0 && N < 16, "vmcnt");
  __builtin_amdgcn_s_waitcnt(N | (0x7 << 4) | (0xF << 8));
}
// row index of the K tile that feeds MFMA row i (bits 2 and 3 swapped)
__device__ __forceinline__ int fp_perm(int i) {
  return (i & ~12) | ((i & 4) << 1) | ((i & 8) >> 1);
}

__global__ __launch_bounds__(FP_NW * 64) __attribute__((amdgpu_waves_per_eu(4)))
void k_flash_bf16(const bf16_t* __restrict__ qkv, const bf16_t* __restrict__ vt,
                       bf16_t* __restrict__ out, int n_head) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  constexpr int S = 2;                             // LDS stages
  __shared__ __attribute__((aligned(16))) bf16_t Ks[S][FP_KT * 64];   // [key][dim]
  __shared__ __attribute__((aligned(16))) bf16_t Vs[S][64 * FP_KT];   // [dim][key]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // XCD-aware work order: the hardware deals blocks round-robin to the 8
  // XCDs in dispatch order (x fastest), so block i runs on XCD i % 8.  Each
  // XCD takes a contiguous range of (query block, head, clip) work items,
  // query block fastest, so the query blocks of one (clip, head) share an
  // L2 and its K and V^T tiles are fetched from beyond it about once.
  int qb, h, b;
  {
    const int nqb = gridDim.x, nh = gridDim.y;
    const int total = nqb * nh * (int)gridDim.z;
    const int lin = (int)blockIdx.x + nqb * ((int)blockIdx.y + nh * (int)blockIdx.z);
    const int per = total / 8, rem = total % 8, xcd = lin % 8;
    const int w = xcd * per + min(xcd, rem) + lin / 8;
    qb = w % nqb;
    h = (w / nqb) % nh;
    b = w / (nqb * nh);
  }
  const int d = n_head * 64, ld3 = 3 * d;
  const bf16_t* base = qkv + (int64_t)b * kCtx * ld3;
  const int half = lane >> 5, l32 = lane & 31;
  const int q = qb * (FP_NW * 32) + wave * 32 + l32;   // this lane's query
  constexpr int NT = (kCtx + FP_KT - 1) / FP_KT;

  // Q fragments (B operand of S^T): dims kk*16 + half*8 .. +8 of query q
  bf16x8 qf[4];
  {
    const bf16_t* qp = base + (int64_t)(q < kCtx ? q : 0) * ld3 + h * 64 + half * 8;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      uint4 v = {0u, 0u, 0u, 0u};
      if (q < kCtx) v = *(const uint4*)(qp + kk * 16);
      qf[kk] = as_bf16x8(v);
    }
  }

  // Direct loads: wave w fills rows 8w .. 8w+7 of both tiles; lane l lands
  // 16 bytes at slot l % 8 of row 8w + l / 8 and fetches the chunk that the
  // swizzle puts there.  K rows past position 1499 re-read row 1499 (their
  // scores are masked); V^T rows are padded to kVtLd >= 64 NT positions.
  const int lrow = wave * 8 + (lane >> 3);
  const int lch = (lane & 7) ^ ((lrow >> 1) & 7);
  const uint32_t k_lds = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) bf16_t*)&Ks[0][0] + (uint32_t)(wave * 1024));
  const uint32_t v_lds = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) bf16_t*)&Vs[0][0] + (uint32_t)(wave * 1024));
  const bf16_t* kbase = base + d + h * 64;                          // K columns of head h
  const bf16_t* vbase = vt + ((int64_t)b * n_head + h) * 64 * kVtLd;
  const uint32_t v_off = (uint32_t)((lrow * kVtLd + lch * 8) * 2);
  auto issue = [&](int t) {
    const int k0 = t * FP_KT;
    const int key = min(k0 + lrow, kCtx - 1);
    const uint32_t so = (uint32_t)((t % S) * FP_KT * 64 * 2);
    fp_dma16(k_lds + so, (uint32_t)((key * ld3 + lch * 8) * 2), kbase);
    fp_dma16(v_lds + so, v_off, vbase + k0);
  };

  // fragment read offsets (elements) within a stage
  const int sw = (l32 >> 1) & 7;                       // swizzle of rows l32 and 32 + l32
  int koff[2][4];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int row = kb * 32 + fp_perm(l32);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) koff[kb][kk] = row * 64 + (((kk * 2 + half) ^ ((row >> 1) & 7)) * 8);
  }

  f32x16 zero16;
#pragma unroll
  for (int r = 0; r < 16; ++r) zero16[r] = 0.f;
  // all eight K fragments in flight before the first MFMA needs one
  // scores of tile t: four K fragments in flight per 32-key block
  auto scores = [&](int t, f32x16 (&s)[2]) {
    const bf16_t* Kc = Ks[t % S];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      bf16x8 kf[4];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) kf[kk] = *(const bf16x8*)(Kc + koff[kb][kk]);
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf[kk],
                                                        kk == 0 ? zero16 : s[kb], 0, 0, 0);
    }
  };

  f32x16 o0, o1;                                   // O^T dims 0..31, 32..63
#pragma unroll
  for (int r = 0; r < 16; ++r) o0[r] = o1[r] = 0.f;
  float m = 0.f, l = 0.f;
  bool zref = true;                                // every lane of the wave has m == 0
  const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3F803F80u);

  // softmax of tile t's scores (in s) and its P V product
  // (the rare branches carry an empty volatile asm so that the compiler
  // keeps them as branches instead of executing them on every tile)
  auto consume = [&](int t, f32x16 (&s)[2]) {
    const int k0 = t * FP_KT;
    // V fragments: chunk kb*4 + hf*2 + half of V^T rows l32 and 32 + l32
    const bf16_t* Vc = Vs[t % S];
    auto vfrag = [&](int kb, int hf, int row) {
      return *(const bf16x8*)(Vc + row * 64 + (((kb * 4 + hf * 2 + half) ^ sw) * 8));
    };
    if (!zref) {                                   // wave-uniform: some lane's m moved
      asm volatile("");
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kb][r] -= m;
    }
    if (k0 + FP_KT > kCtx) {                       // last tile: keys past 1500 do not exist
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k0 + kb * 32 + (r >> 3) * 16 + half * 8 + (r & 7);
          if (key >= kCtx) s[kb][r] = -INFINITY;
        }
    }
    // probabilities of the tile against the current reference, packed to
    // bf16 (the P V product's B operand), and their sum
    uint32_t u[2][2][4];
    float lt = 0.f;
    auto probs = [&]() {
      float ls[4] = {0.f, 0.f, 0.f, 0.f};          // four independent sum chains
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            // keys kb*32 + hf*16 + half*8 + 2i, +1: registers hf*8 + 2i, +1
            u[kb][hf][i] = pack2_bf16(__builtin_amdgcn_exp2f(s[kb][hf * 8 + 2 * i]),
                                      __builtin_amdgcn_exp2f(s[kb][hf * 8 + 2 * i + 1]));
            ls[i] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, u[kb][hf][i]),
                                                    ones, ls[i], false);
          }
      lt = (ls[0] + ls[1]) + (ls[2] + ls[3]);
    };
    probs();
    // Lazy reference: probabilities are exp2(s - m) with m = 0 as long as
    // every score of the wave stays within 2^6 of it, so the common case
    // needs no subtraction at all.  exp2(s - m) may then reach 2^64, which
    // fp32 sums and bf16 operands carry with unchanged relative precision
    // (both reach 2^127); the final 1/l cancels the offset.  The common case
    // does not look for the tile's maximum either: a score more than 2^6
    // above m (or +inf) makes its lane's probability sum exceed 2^64, and on
    // the first tile a lane whose scores all lie far below 0 sums to less
    // than 2^-64.  Only such tiles take the exact maximum: a first tile whose
    // maximum lies outside [-64, 64] sets m to it; a later maximum more than
    // 2^6 above m moves m up and rescales O and l; the tile's probabilities
    // are then recomputed.
    if (__any(lt > 0x1p64f) || (t == 0 && __any(lt < 0x1p-64f))) {
      asm volatile("");
      float tmax = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, s[kb][r]);
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
      if (t == 0) {
        if (__any(fabsf(tmax) > 64.0f)) {          // 64 real keys: finite
          m = tmax;
          zref = false;
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) s[kb][r] -= tmax;
        }
      } else if (__any(tmax > 64.0f)) {
        const float shift = fmaxf(tmax, 0.f);
        const float alpha = __builtin_amdgcn_exp2f(-shift);
        m += shift;
        zref = false;
        l *= alpha;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          o0[r] *= alpha;
          o1[r] *= alpha;
        }
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) s[kb][r] -= shift;
      }
      probs();
    }
    l += lt;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const bf16x8 pb = as_bf16x8(uint4{u[kb][hf][0], u[kb][hf][1], u[kb][hf][2], u[kb][hf][3]});
        o0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfrag(kb, hf, l32), pb, o0, 0, 0, 0);
        o1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfrag(kb, hf, 32 + l32), pb, o1, 0, 0, 0);
      }
  };

  // tile t+1 loads while tile t is consumed
  f32x16 sc[2];
  issue(0);
  for (int t = 0; t < NT; ++t) {
    fp_wait_vmcnt<0>();                            // tile t landed
    __syncthreads();                               // ... for every wave; tile t-1's stage free
    if (t + 1 < NT) issue(t + 1);
    scores(t, sc);
    consume(t, sc);
  }
  l += __shfl_xor(l, 32, 64);
  if (q >= kCtx) return;
  const float inv = 1.0f / l;
  bf16_t* op = out + ((int64_t)b * kCtx + q) * d + h * 64;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int d0 = g * 8 + half * 4;
    uint2 w0 = {pack2_bf16(o0[g * 4 + 0] * inv, o0[g * 4 + 1] * inv),
                pack2_bf16(o0[g * 4 + 2] * inv, o0[g * 4 + 3] * inv)};
    uint2 w1 = {pack2_bf16(o1[g * 4 + 0] * inv, o1[g * 4 + 1] * inv),
                pack2_bf16(o1[g * 4 + 2] * inv, o1[g * 4 + 3] * inv)};
    *(uint2*)(op + d0) = w0;
    *(uint2*)(op + 32 + d0) = w1;
  }
}

void flash_attn_bf16(const bf16_t* qkv, const bf16_t* vt, bf16_t* out, int B, int n_head,
                     hipStream_t s) {
  if (B <= 0) return;
  static_assert(kVtLd >= FP_KT * ((kCtx + FP_KT - 1) / FP_KT), "V^T rows cover every tile");
  dim3 grid((kCtx + FP_NW * 32 - 1) / (FP_NW * 32), n_head, B);
  k_flash_bf16<<<grid, FP_NW * 64, 0, s>>>(qkv, vt, out, n_head);
}

// Lays given q / k / v ([B*1500][d] float32) out as the encoder attention
// kernels read them: which = 0, 1 -> columns 0..d-1, d..2d-1 of qkv (q times
// qmul); which = 2 -> columns 2d..3d-1 (fp32), or V^T [b][h][dim][kVtLd]
// (bf16).
template <typename T>
__global__ void k_pack_attn_operand(const float* __restrict__ src, int which, int rows, int d,
                                    int n_head, float qmul, T* __restrict__ qkv,
                                    T* __restrict__ vt) {
  const int64_t n = (int64_t)rows * d;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / d;
    const int c = (int)(i - r * d);
    const float x = which == 0 ? src[i] * qmul : src[i];
    if (which < 2 || vt == nullptr) {
      St<T>::st(qkv, r * 3 * d + which * d + c, x);
    } else {
      const int64_t g = r / kCtx, t = r - g * kCtx;
      St<T>::st(vt, ((g * n_head + (c >> 6)) * kHeadDim + (c & 63)) * kVtLd + t, x);
    }
  }
}
template <typename T>
void pack_attn_operand(const float* src, int which, int rows, int d, int n_head, float qmul,
                       T* qkv, T* vt, hipStream_t s) {
  const int64_t n = (int64_t)rows * d;
  if (n <= 0) return;
  const int grid = (int)std::min<int64_t>((n + 255) / 256, 65536);
  k_pack_attn_operand<T><<<grid, 256, 0, s>>>(src, which, rows, d, n_head, qmul, qkv, vt);
}
template void pack_attn_operand<float>(const float*, int, int, int, int, float, float*, float*,
                                       hipStream_t);
template void pack_attn_operand<bf16_t>(const float*, int, int, int, int, float, bf16_t*,
                                        bf16_t*, hipStream_t);

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
// Keys per block of the decode attention: a row's keys are split into chunks
// of DA_CK handled by separate blocks (flash-decoding), which fills the chip
// in whole rounds (128 rows x 20 heads x 4 chunks of the 1500 cross keys =
// 10240 blocks = 5 rounds of 2048 resident blocks); a combine kernel merges
// the chunks' (max, sum, weighted values).
constexpr int DA_CK = 384;

// SELF: queries, keys and values of the step come from the fused QKV output
// `src` [D][3d].  Cross: the query is bias + the q_splits float32 partial
// sums of the query product (q_part[s][row][d]).
template <typename T, bool SELF>
__global__ __launch_bounds__(256) void k_decode_attn(const T* __restrict__ src,
                                                     const float* __restrict__ q_part,
                                                     int q_splits, const float* __restrict__ q_bias,
                                                     int D, T* cache,
                                                     int64_t slot_stride, int64_t layer_off,
                                                     const int32_t* slots, const int32_t* pos,
                                                     int n_head, float* __restrict__ part) {
  constexpr int CTX = SELF ? kTextCtx : kCtx;
  __shared__ float qs[64];
  __shared__ float sc[DA_CK];
  __shared__ float red[4];
  __shared__ float ored[4][64];
  const int h = blockIdx.x, row = blockIdx.y, chunk = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = n_head * 64;
  const int ldsrc = 3 * d;
  const int n = SELF ? pos[row] + 1 : kCtx;
  const int k0 = chunk * DA_CK;
  if (k0 >= n) return;                          // this row has fewer chunks (uniform per block)
  const int kn = min(DA_CK, n - k0);            // keys of this chunk
  const int slot = slots[row];
  T* kb = cache + (int64_t)slot * slot_stride + layer_off + (int64_t)h * CTX * 64;
  T* vb = kb + (int64_t)n_head * CTX * 64;
  const T* srow = SELF ? src + (int64_t)row * ldsrc + h * 64 : nullptr;

  if (tid < 64) {
    if constexpr (SELF) {
      qs[tid] = St<T>::ld(srow, tid) * 0.125f;
    } else {
      const int c = h * 64 + tid;
      float v = q_bias[c];
      for (int sp = 0; sp < q_splits; ++sp) v += q_part[((int64_t)sp * D + row) * d + c];
      qs[tid] = v * 0.125f;
    }
  }
  if (SELF && tid < 128 && n - 1 >= k0 && n - 1 < k0 + kn) {
    // the chunk holding position n-1 stores this step's k, v there
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

  // scores of the chunk's keys (8 lanes per key, 16-byte loads)
  for (int g0 = 0; g0 < kn; g0 += 128) {
    float partial[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int kk = g0 + u * 32 + wave * 8 + sub, key = k0 + kk;
      partial[u] = 0.f;
      if (kk < kn) {
        const T* kp = (SELF && key == n - 1) ? (srow + d) : (kb + (int64_t)key * 64);
        float kv[8];
        load8(kp + dc, kv);
#pragma unroll
        for (int i = 0; i < 8; ++i) partial[u] = fmaf(qv[i], kv[i], partial[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      float p = partial[u];
      p += __shfl_xor(p, 1, 64);
      p += __shfl_xor(p, 2, 64);
      p += __shfl_xor(p, 4, 64);
      const int kk = g0 + u * 32 + wave * 8 + sub;
      if ((lane & 7) == 0 && kk < kn) sc[kk] = p;
    }
  }
  __syncthreads();

  float mx = -INFINITY;
  for (int k = tid; k < kn; k += 256) mx = fmaxf(mx, sc[k]);
  mx = wave_max(mx);
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float sum = 0.f;
  for (int k = tid; k < kn; k += 256) {
    float p = expf(sc[k] - mx);
    sc[k] = p;
    sum += p;
  }
  sum = wave_sum(sum);
  if (lane == 0) red[wave] = sum;
  __syncthreads();
  const float l = red[0] + red[1] + red[2] + red[3];

  // probability-weighted values of the chunk
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  for (int g0 = 0; g0 < kn; g0 += 128) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int kk = g0 + u * 32 + wave * 8 + sub, key = k0 + kk;
      if (kk < kn) {
        const T* vp = (SELF && key == n - 1) ? (srow + 2 * d) : (vb + (int64_t)key * 64);
        float vv[8];
        load8(vp + dc, vv);
        const float p = sc[kk];
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
  // partial record of (row, head, chunk): [max, sum, 64 weighted values]
  float* rec = part + (((int64_t)row * n_head + h) * DA_NCH + chunk) * DA_REC;
  if (tid < 64) rec[2 + tid] = ored[0][tid] + ored[1][tid] + ored[2][tid] + ored[3][tid];
  if (tid == 0) {
    rec[0] = mx;
    rec[1] = l;
  }
}

// out[row][h] = sum_c e^{m_c - M} acc_c / sum_c e^{m_c - M} l_c over the
// row's chunks (M = max_c m_c).  One wave per (row, head).
template <typename T, bool SELF>
__global__ __launch_bounds__(256) void k_decode_combine(const float* __restrict__ part,
                                                        const int32_t* pos, int D, int n_head,
                                                        T* __restrict__ out) {
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (w >= D * n_head) return;
  const int row = w / n_head, h = w - row * n_head;
  const int n = SELF ? pos[row] + 1 : kCtx;
  const int nch = (n + DA_CK - 1) / DA_CK;
  const float* rec = part + (int64_t)w * DA_NCH * DA_REC;
  float M = -INFINITY;
  for (int c = 0; c < nch; ++c) M = fmaxf(M, rec[c * DA_REC]);
  float num = 0.f, den = 0.f;
  for (int c = 0; c < nch; ++c) {
    const float f = expf(rec[c * DA_REC] - M);
    den += f * rec[c * DA_REC + 1];
    num += f * rec[c * DA_REC + 2 + lane];
  }
  St<T>::st(out, (int64_t)row * n_head * 64 + h * 64 + lane, num / den);
}

// bf16 decode cross attention with every K and V row of the block's keys
// in flight at once: each thread issues the 16-byte loads of its share of
// all keys (8 lanes per key, 32 keys per pass, NP passes) for K and V before
// any arithmetic, so the value stream's latency hides behind the scores and
// the softmax; scores stay in registers (one cross-lane reduction per key),
// and three block barriers remain.  The query is the bias plus the qp_splits
// float32 partial sums of its product (qp[s][row][d]).  One block per (row,
// head, 384-key chunk), leaving a (max, sum, weighted values) record for
// the combine kernel.
template <int NP>
__global__ __launch_bounds__(256) void k_dattn_cross_bf16(const float* __restrict__ qp, int qp_splits,
                                                          const float* __restrict__ qp_bias, int D,
                                                          const bf16_t* cache, int64_t slot_stride,
                                                          int64_t layer_off, const int32_t* slots,
                                                          int n_head, float* __restrict__ part) {
  constexpr int CK = NP * 32;                       // keys per block
  __shared__ float qs[64];
  __shared__ float red[2][4];
  __shared__ float ored[4][64];
  const int h = blockIdx.x, row = blockIdx.y, chunk = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = n_head * 64;
  const int k0 = chunk * CK;
  const int kn = min(CK, kCtx - k0);
  const int slot = slots[row];
  const bf16_t* kb = cache + (int64_t)slot * slot_stride + layer_off + (int64_t)h * kCtx * 64;
  const bf16_t* vb = kb + (int64_t)n_head * kCtx * 64;
  const int sub = lane >> 3, dc = (lane & 7) * 8;

  // all loads of the block's keys first
  uint4 kr[NP], vr[NP];
  const uint4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int kk = p * 32 + wave * 8 + sub, key = k0 + kk;
    kr[p] = zero;
    vr[p] = zero;
    if (kk < kn) {
      kr[p] = *(const uint4*)(kb + (int64_t)key * 64 + dc);
      vr[p] = *(const uint4*)(vb + (int64_t)key * 64 + dc);
    }
  }
  if (tid < 64) {
    const int c = h * 64 + tid;
    float v = qp_bias[c];
    for (int sp = 0; sp < qp_splits; ++sp) v += qp[((int64_t)sp * D + row) * d + c];
    qs[tid] = v * 0.125f;
  }
  __syncthreads();
  float qv[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) qv[i] = qs[dc + i];

  // scores: 8 dims per lane, summed over the key's 8 lanes
  float sc[NP];
  float mx = -INFINITY;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    float kv[8];
    load8((const bf16_t*)&kr[p], kv);
    float a = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) a = fmaf(qv[i], kv[i], a);
    a += __shfl_xor(a, 1, 64);
    a += __shfl_xor(a, 2, 64);
    a += __shfl_xor(a, 4, 64);
    const int kk = p * 32 + wave * 8 + sub;
    sc[p] = kk < kn ? a : -INFINITY;
    mx = fmaxf(mx, sc[p]);
  }
  mx = wave_max(mx);
  if (lane == 0) red[0][wave] = mx;
  __syncthreads();
  const float M = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));

  // probabilities and the weighted value sum
  float l = 0.f, acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const float pr = expf(sc[p] - M);                // 0 for keys past the chunk
    l += pr;
    float vv[8];
    load8((const bf16_t*)&vr[p], vv);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = fmaf(pr, vv[i], acc[i]);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float a = acc[i];
    a += __shfl_xor(a, 8, 64);
    a += __shfl_xor(a, 16, 64);
    a += __shfl_xor(a, 32, 64);
    acc[i] = a;
  }
  // each key's probability was added by its 8 lanes
  l = wave_sum(l) * 0.125f;
  if (lane < 8) {
#pragma unroll
    for (int i = 0; i < 8; ++i) ored[wave][dc + i] = acc[i];
  }
  if (lane == 0) red[1][wave] = l;
  __syncthreads();
  if (tid < 64) {
    float* rec = part + (((int64_t)row * n_head + h) * DA_NCH + chunk) * DA_REC;
    rec[2 + tid] = ored[0][tid] + ored[1][tid] + ored[2][tid] + ored[3][tid];
    if (tid == 0) {
      rec[0] = M;
      rec[1] = red[1][0] + red[1][1] + red[1][2] + red[1][3];
    }
  }
}

// bf16 decode self attention: one block per (row, head) over the row's
// position + 1 keys, writing the output directly.  The keys go in two halves
// of DS_NP passes (224 keys) each, so a thread holds only one half's K and V
// rows (about 90 VGPRs: five blocks per CU, which is what the short rows'
// latency needs); the second half, present only for rows longer than 224
// keys, loads its keys as soon as the first half's scores are done and its
// values once the first half's weighted sum is, and joins through the usual
// online-softmax rescale (block-wide maxima, so all lanes share one
// reference).  The query, key and value of the step are bias + the
// qp_splits float32 partial sums of the QKV product (qp[s][row][3d]); the new
// key and value, rounded to bf16, go into the cache at the last position and
// into the scores from LDS.
constexpr int DS_NP = 7;
constexpr int DS_HALF = DS_NP * 32;
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(5))) void k_dattn_self_bf16(const float* __restrict__ qp, int qp_splits,
                                                         const float* __restrict__ qp_bias, int D,
                                                         bf16_t* cache, int64_t slot_stride,
                                                         int64_t layer_off, const int32_t* slots,
                                                         const int32_t* pos, int n_head,
                                                         bf16_t* __restrict__ out) {
  static_assert(2 * DS_HALF >= kTextCtx, "two halves cover the decoder context");
  __shared__ float qs[64];
  __shared__ __attribute__((aligned(16))) bf16_t kvnew[2][64];
  __shared__ float red[3][4];
  __shared__ float ored[4][64];
  const int h = blockIdx.x, row = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = n_head * 64;
  const int n = pos[row] + 1;                       // keys, this step's included
  const int slot = slots[row];
  bf16_t* kb = cache + (int64_t)slot * slot_stride + layer_off + (int64_t)h * kTextCtx * 64;
  bf16_t* vb = kb + (int64_t)n_head * kTextCtx * 64;
  const int sub = lane >> 3, dc = (lane & 7) * 8;
  const bool two = n > DS_HALF;                     // block-uniform
  auto key_of = [&](int hf, int p) { return hf * DS_HALF + p * 32 + wave * 8 + sub; };

  // cached keys (all but the last) of a half
  uint4 kr[DS_NP], vr[DS_NP];
  const uint4 zero = {0u, 0u, 0u, 0u};
  auto load_k = [&](int hf) {
#pragma unroll
    for (int p = 0; p < DS_NP; ++p) {
      const int key = key_of(hf, p);
      kr[p] = zero;
      if (key < n - 1) kr[p] = *(const uint4*)(kb + (int64_t)key * 64 + dc);
    }
  };
  auto load_v = [&](int hf) {
#pragma unroll
    for (int p = 0; p < DS_NP; ++p) {
      const int key = key_of(hf, p);
      vr[p] = zero;
      if (key < n - 1) vr[p] = *(const uint4*)(vb + (int64_t)key * 64 + dc);
    }
  };
  load_k(0);
  load_v(0);
  // query, new key and value: bias + the product's partials
  if (tid < 192) {
    const int part_i = tid >> 6, j = tid & 63;       // 0: q, 1: k, 2: v
    const int c = part_i * d + h * 64 + j;
    float v = qp_bias[c];
    for (int sp = 0; sp < qp_splits; ++sp) v += qp[((int64_t)sp * D + row) * 3 * d + c];
    if (part_i == 0) {
      qs[j] = v * 0.125f;
    } else {
      const bf16_t b = f2bf(v);
      kvnew[part_i - 1][j] = b;
      (part_i == 1 ? kb : vb)[(int64_t)(n - 1) * 64 + j] = b;
    }
  }
  __syncthreads();
  float qv[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) qv[i] = qs[dc + i];

  float M = -INFINITY, l = 0.f, acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
  auto half = [&](int hf) {
#pragma unroll
    for (int p = 0; p < DS_NP; ++p)
      if (key_of(hf, p) == n - 1) {
        kr[p] = *(const uint4*)&kvnew[0][dc];
        vr[p] = *(const uint4*)&kvnew[1][dc];
      }
    float sc[DS_NP];
    float mx = -INFINITY;
#pragma unroll
    for (int p = 0; p < DS_NP; ++p) {
      float kv[8];
      load8((const bf16_t*)&kr[p], kv);
      float a = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) a = fmaf(qv[i], kv[i], a);
      a += __shfl_xor(a, 1, 64);
      a += __shfl_xor(a, 2, 64);
      a += __shfl_xor(a, 4, 64);
      sc[p] = key_of(hf, p) < n ? a : -INFINITY;
      mx = fmaxf(mx, sc[p]);
    }
    mx = wave_max(mx);
    if (lane == 0) red[hf][wave] = mx;
    __syncthreads();
    if (hf == 0 && two) load_k(1);                   // the first half's keys are done with
    const float Mn = fmaxf(M, fmaxf(fmaxf(red[hf][0], red[hf][1]), fmaxf(red[hf][2], red[hf][3])));
    const float f = expf(M - Mn);                    // 0 on the first half (M = -inf)
    l *= f;
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] *= f;
#pragma unroll
    for (int p = 0; p < DS_NP; ++p) {
      const float pr = expf(sc[p] - Mn);             // 0 for keys past the row
      l += pr;
      float vv[8];
      load8((const bf16_t*)&vr[p], vv);
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] = fmaf(pr, vv[i], acc[i]);
    }
    M = Mn;
    if (hf == 0 && two) load_v(1);                   // ... and so are its values
  };
  half(0);
  if (two) half(1);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float a = acc[i];
    a += __shfl_xor(a, 8, 64);
    a += __shfl_xor(a, 16, 64);
    a += __shfl_xor(a, 32, 64);
    acc[i] = a;
  }
  // each key's probability was added by its 8 lanes
  l = wave_sum(l) * 0.125f;
  if (lane < 8) {
#pragma unroll
    for (int i = 0; i < 8; ++i) ored[wave][dc + i] = acc[i];
  }
  if (lane == 0) red[2][wave] = l;
  __syncthreads();
  if (tid < 64) {
    const float o = ored[0][tid] + ored[1][tid] + ored[2][tid] + ored[3][tid];
    const float L = red[2][0] + red[2][1] + red[2][2] + red[2][3];
    out[(int64_t)row * d + h * 64 + tid] = f2bf(o / L);
  }
}

int decode_attn_part_floats(int D, int n_head) { return D * n_head * DA_NCH * DA_REC; }

template <typename T>
void decode_self_attn(const T* qkv, const float* qkv_part, int qkv_splits, const float* qkv_bias,
                      T* cache, int64_t slot_stride, int64_t layer_off, const int32_t* slots,
                      const int32_t* pos, int D, int n_head, T* out, float* part,
                      hipStream_t s) {
  if (D <= 0) return;
  if constexpr (sizeof(T) == 2) {
    k_dattn_self_bf16<<<dim3(n_head, D, 1), 256, 0, s>>>(
        qkv_part, qkv_splits, qkv_bias, D, (bf16_t*)cache, slot_stride, layer_off, slots, pos,
        n_head, (bf16_t*)out);
    return;
  }
  constexpr int nch = (kTextCtx + DA_CK - 1) / DA_CK;
  k_decode_attn<T, true><<<dim3(n_head, D, nch), 256, 0, s>>>(
      qkv, nullptr, 0, nullptr, D, cache, slot_stride, layer_off, slots, pos, n_head, part);
  k_decode_combine<T, true><<<(D * n_head + 3) / 4, 256, 0, s>>>(part, pos, D, n_head, out);
}
template <typename T>
void decode_cross_attn(const float* q_part, int q_splits, const float* q_bias, T* cache,
                       int64_t slot_stride, int64_t layer_off, const int32_t* slots, int D,
                       int n_head, T* out, float* part, hipStream_t s) {
  if (D <= 0) return;
  constexpr int nch = (kCtx + DA_CK - 1) / DA_CK;
  if constexpr (sizeof(T) == 2) {
    static_assert(DA_CK % 32 == 0, "passes");
    k_dattn_cross_bf16<DA_CK / 32><<<dim3(n_head, D, nch), 256, 0, s>>>(
        q_part, q_splits, q_bias, D, (const bf16_t*)cache, slot_stride, layer_off, slots, n_head,
        part);
    k_decode_combine<T, false><<<(D * n_head + 3) / 4, 256, 0, s>>>(part, nullptr, D, n_head, out);
    return;
  }
  k_decode_attn<T, false><<<dim3(n_head, D, nch), 256, 0, s>>>(
      nullptr, q_part, q_splits, q_bias, D, cache, slot_stride, layer_off, slots, nullptr, n_head,
      part);
  k_decode_combine<T, false><<<(D * n_head + 3) / 4, 256, 0, s>>>(part, nullptr, D, n_head, out);
}
template void decode_self_attn<float>(const float*, const float*, int, const float*, float*,
                                      int64_t, int64_t, const int32_t*, const int32_t*, int, int,
                                      float*, float*, hipStream_t);
template void decode_self_attn<bf16_t>(const bf16_t*, const float*, int, const float*, bf16_t*,
                                       int64_t, int64_t, const int32_t*, const int32_t*, int, int,
                                       bf16_t*, float*, hipStream_t);
template void decode_cross_attn<float>(const float*, int, const float*, float*, int64_t,
                                       int64_t, const int32_t*, int, int, float*, float*,
                                       hipStream_t);
template void decode_cross_attn<bf16_t>(const float*, int, const float*, bf16_t*, int64_t,
                                        int64_t, const int32_t*, int, int, bf16_t*, float*,
                                        hipStream_t);

}  // namespace asr
