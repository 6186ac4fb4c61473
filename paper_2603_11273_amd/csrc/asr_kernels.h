// Internal declarations shared by the HIP kernels and the runtime.
// Not part of the public ABI (include/asr.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace asr {

constexpr int kSampleRate = 16000;
constexpr int kSamples30s = 480000;   // one encoder segment
constexpr int kNFFT = 400;
constexpr int kHop = 160;
constexpr int kBins = kNFFT / 2 + 1;  // 201
constexpr int kFrames = 3000;
constexpr int kCtx = 1500;            // encoder positions
constexpr int kTextCtx = 448;         // decoder positions
constexpr int kHeadDim = 64;

// Storage tags: float32 or bfloat16 (raw 16-bit pattern).
typedef uint16_t bf16_t;

// ---------------------------------------------------------------------------
// Launch parameter blocks
// ---------------------------------------------------------------------------

// A operand of C = A . W^T: row r of the logical A lives at
//   A + (r / rows_per_batch) * batch_stride + (r % rows_per_batch) * lda
// (elements), which expresses both plain row-major matrices and the implicit
// im2col windows of the two stem convolutions.
struct AView {
  const void* ptr;
  int64_t lda;
  int64_t batch_stride;
  int32_t rows_per_batch;
};

enum EpiKind : int32_t {
  EPI_STORE = 0,      // out[r][n] = acc + bias[n]                       (storage type)
  EPI_GELU = 1,       // out[r][n] = gelu(acc + bias[n])                 (storage type)
  EPI_CONV1 = 3,      // h1[g][t+1][n] = gelu(acc + bias[n]); h1[g][0][n] = 0 (storage)
  EPI_CONV2 = 4,      // x[r][n] = gelu(acc + bias[n]) + pos[r % 1500][n]   (float32)
  EPI_XKV = 5,        // cross cache of slot[g], all decoder layers        (storage)
  EPI_QKV = 6,        // q (x kQScaleLog2), k -> out[r][n] (n < 2d); v -> out2 = V^T (storage)
};

// EPI_QKV stores q multiplied by 1/sqrt(64) * log2(e): the encoder's flash
// attention then works in the exp2 domain without a per-score multiply.
constexpr float kQScaleLog2 = 0.125f * 1.4426950408889634f;

// Row stride (positions) of the per-head transposed V written by EPI_QKV:
// V^T[b][h][dim][kVtLd], positions 1500..1535 stay zero.
constexpr int kVtLd = 1536;

struct Epilogue {
  int32_t kind;
  void* out;            // destination (type depends on kind)
  int64_t ldc;          // row stride of out (elements) for STORE/GELU/CONV2/QKV
  const float* bias;    // [N]
  const float* pos;     // CONV2: sinusoid table [1500][N]
  const int32_t* slots; // XKV: slot of each clip
  int64_t slot_stride;  // XKV: elements per slot's cross cache
  int32_t d_model;      // XKV / CONV1 / QKV
  int32_t n_head;       // XKV / QKV
  void* out2;           // QKV: transposed V [B][H][64][kVtLd]
};

// Dense GEMM C[M][N] = A[M][K] . W[N][K]^T with a fused epilogue.
void gemm_bf16(const AView& a, const bf16_t* w, int M, int N, int K, const Epilogue& e,
               hipStream_t s);
void gemm_f32(const AView& a, const float* w, int M, int N, int K, const Epilogue& e,
              hipStream_t s);

// Number of CUs the persistent bf16 GEMM leaves free (process-wide; 0 = none).
void gemm_set_cu_reserve(int n);

// Skinny GEMM for decode rows (D <= 128, N % 32 == 0, K % 64 == 0), x [D][K]
// times w [N][K]^T.  DG_PARTIAL: out = float32 partial sums over K slices,
// partial[s][b][n] for s < dgemm_splits(N, K) (returned); DG_BIAS / DG_GELU:
// out[b][n] = (gelu)(sum + bias[n]) in bf16 (returns 1).
enum DgEpi : int32_t { DG_PARTIAL = 0, DG_BIAS = 1, DG_GELU = 2 };
int dgemm_bf16(const bf16_t* x, const bf16_t* w, int D, int N, int K, int epi,
               const float* bias, void* out, hipStream_t s);
int dgemm_splits(int N, int K);
// fp32 path: out[b][n] = sum_k x[b][k] w[n][k] (one partial slice, no bias).
void dgemm_f32(const float* x, const float* w, int D, int N, int K, float* out, hipStream_t s);
// out = epilogue(sum_s partial[s] + bias): mode 0 store (T), 1 gelu (T), 2 residual add (f32).
template <typename T>
void dgemm_reduce(const float* partial, int splits, int D, int N, const float* bias, int mode,
                  void* out, hipStream_t s);

// h[b] += bias + sum_s partial[s][b]; xn[b] = LayerNorm(h[b]) with (g, beta).  d <= 2048.
template <typename T>
void reduce_resid_ln(const float* partial, int splits, int D, int d, const float* bias, float* h,
                     const float* g, const float* beta, T* xn, hipStream_t s);

// Vocabulary projection fused with argmax: keys[b][tile] (ordered value, lowest index).
void vocab_argmax_bf16(const bf16_t* x, const bf16_t* emb, int D, int V, int K,
                       uint64_t* keys, int n_tiles, float* logits, hipStream_t s);
void vocab_logits_f32(const float* x, const float* emb, int D, int V, int K, float* logits,
                      hipStream_t s);
void logits_argmax_keys(const float* logits, int D, int V, uint64_t* keys, int n_tiles,
                        hipStream_t s);
void argmax_finish(const uint64_t* keys, int D, int n_tiles, int32_t* out, int32_t* nan_flag,
                   hipStream_t s);
int vocab_tiles(int V);

// LayerNorm rows of a float32 matrix into storage type T.
template <typename T>
void layer_norm(const float* x, int rows, int d, const float* g, const float* b, T* out,
                hipStream_t s);
// Residual add fused with the LayerNorm that follows it, the branches in
// storage type T (rows ldy elements apart), the stream x in float32:
//   y2 == nullptr, store:  x += y1,            out = LN(x)
//   y2 == nullptr, !store: out = LN(x + y1)    (x unchanged)
//   y2 != nullptr:         x = (x + y1) + y2,  out = LN(x)
template <typename T>
void residual_layer_norm(float* x, const T* y1, const T* y2, int64_t ldy, bool store, int rows,
                         int d, const float* g, const float* b, T* out, hipStream_t s);

// Writes given float32 operands [B*1500][d] where the attention kernels read
// them (which: 0 = q, scaled by qmul; 1 = k; 2 = v, transposed into vt for
// bf16, else columns 2d.. of qkv).
template <typename T>
void pack_attn_operand(const float* src, int which, int rows, int d, int n_head, float qmul,
                       T* qkv, T* vt, hipStream_t s);
// Encoder self-attention over 1500 positions, qkv [B*1500][3d], out [B*1500][d].
void flash_attn_bf16(const bf16_t* qkv, const bf16_t* vt, bf16_t* out, int B, int n_head,
                     hipStream_t s);
void flash_attn_f32(const float* qkv, float* out, int B, int n_head, hipStream_t s);

// Decode attention.  Self: writes k, v of each row at its slot position, then
// attends over position + 1 keys.  Cross: attends over 1500 cached keys.
// Keys are split into chunks handled by separate blocks; `part` (at least
// decode_attn_part_floats(D, n_head) floats) holds the per-chunk partials
// that a combine kernel merges into out.
constexpr int DA_NCH = 4;    // chunks per row at most (1500 cross keys / 384)
constexpr int DA_REC = 66;   // floats per partial: max, sum, 64 weighted values
int decode_attn_part_floats(int D, int n_head);
// Self: fp32 contexts read q, k, v from the fused QKV output qkv [D][3d];
// bf16 contexts from the float32 partial sums of the QKV product plus its
// bias (qkv_part[s][b][3d], s < qkv_splits).
template <typename T>
void decode_self_attn(const T* qkv, const float* qkv_part, int qkv_splits, const float* qkv_bias,
                      T* cache, int64_t slot_stride, int64_t layer_off, const int32_t* slots,
                      const int32_t* pos, int D, int n_head, T* out, float* part, hipStream_t s);
// The cross attention takes its queries as the float32 partial sums of the
// query product: q[b] = bias + sum_{s < q_splits} q_part[s][b].
template <typename T>
void decode_cross_attn(const float* q_part, int q_splits, const float* q_bias, T* cache,
                       int64_t slot_stride, int64_t layer_off, const int32_t* slots, int D,
                       int n_head, T* out, float* part, hipStream_t s);

template <typename T>
void embed(const T* tok_emb, const float* pos_emb, const int32_t* tokens, const int32_t* pos,
           int D, int d, float* h, hipStream_t s);

// Log-mel front-end.  pcm_ptrs[i] is a device pointer to clip i's samples.
struct MelTables {
  const float* window;     // [400] periodic Hann
  const float* cos_t;      // [400] cos(2 pi j / 400)
  const float* sin_t;      // [400] sin(2 pi j / 400)
  const float* fb;         // packed nonzero filter weights, filter after filter (<= 402)
  const int32_t* fb_range; // [n_mels][3] first bin, bin count, offset into fb
};
// The front-end transforms kMelGroupFrames consecutive frames of a clip at a
// time and stores each group's largest log-mel value in group_max
// [n_clips][kMelGroups]; mel_normalize reduces a clip's groups to its maximum.
constexpr int kMelGroupFrames = 16;
constexpr int kMelGroups = (kFrames + kMelGroupFrames - 1) / kMelGroupFrames;   // 188
void log_mel(const float* const* pcm_ptrs, const int64_t* n_samples, int n_clips, int n_mels,
             const MelTables& t, float* mel_raw, float* group_max, hipStream_t s);
// The same with the clips' pointers and lengths in the kernel arguments (no
// device-side lists), for up to kMelArgClips clips.
constexpr int kMelArgClips = 64;
struct MelClipArgs {
  const float* ptr[kMelArgClips];
  int64_t n[kMelArgClips];
};
void log_mel_args(const MelClipArgs& clips, int n_clips, int n_mels, const MelTables& t,
                  float* mel_raw, float* group_max, hipStream_t s);
template <typename T>
void mel_normalize(const float* mel_raw, const float* group_max, int n_clips, int n_mels,
                   T* out, int pad_rows, hipStream_t s);

// Utility kernels.
void fill_u32(uint32_t* p, uint32_t v, int64_t n, hipStream_t s);
void fill_f32(float* p, float v, int64_t n, hipStream_t s);
template <typename T>
void convert_from_f32(const float* src, T* dst, int64_t n, hipStream_t s);
template <typename T>
void convert_to_f32(const T* src, float* dst, int64_t n, hipStream_t s);
// dst[o][j][c] = src[o][c][j] for a [d][C][3] conv weight.
template <typename T>
void pack_conv(const float* src, T* dst, int d, int C, hipStream_t s);
// Copies `rows` rows of `cols` floats with strides (elements), converting.
template <typename T>
void copy_rows_from_f32(const float* src, int64_t src_ld, T* dst, int64_t dst_ld, int rows,
                        int cols, hipStream_t s);

}  // namespace asr
