// Runtime behind the C ABI: context, workspace plan, weight packing,
// constant tables, slot bookkeeping, step orchestration and timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "../../include/asr.h"
#include "asr_kernels.h"
#include "queue.h"
#include "serve.h"

using namespace asr;

namespace {

thread_local std::string g_err;

asr_status fail(asr_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

#define HIPCHK(x)                                                                   \
  do {                                                                              \
    hipError_t e_ = (x);                                                            \
    if (e_ != hipSuccess)                                                           \
      return fail(ASR_EDEVICE, std::string(#x) + ": " + hipGetErrorString(e_));     \
  } while (0)

#define CHECK_LAUNCH()                                                              \
  do {                                                                              \
    hipError_t e_ = hipGetLastError();                                              \
    if (e_ != hipSuccess)                                                           \
      return fail(ASR_EDEVICE, std::string("kernel launch: ") + hipGetErrorString(e_)); \
  } while (0)

struct Request {
  int64_t id = 0, arrival_us = 0, n_samples = 0, dur_us = 0;
  int32_t sample_rate = 16000, max_tokens = 448;
  std::vector<float> pcm;             // host copy
  const float* dev_pcm = nullptr;     // caller's device samples
  bool has_audio = false;
};

struct Slot {
  int32_t occupied = 0;
  int64_t id = -1;
  int32_t pos = 0;
  int32_t steps_left = 0;
};

struct EncLayer {
  size_t ln1_g, ln1_b, qkv_w, qkv_b, o_w, o_b, ln2_g, ln2_b, fc1_w, fc1_b, fc2_w, fc2_b;
};
struct DecLayer {
  size_t ln1_g, ln1_b, qkv_w, qkv_b, o_w, o_b, lnx_g, lnx_b, xq_w, xq_b, xo_w, xo_b, ln2_g,
      ln2_b, fc1_w, fc1_b, fc2_w, fc2_b;
};

// How one parameter tensor of the load order lands in device memory.
struct PackOp {
  enum Kind { F32, STORE, CONV } kind;
  size_t dst;      // byte offset
  int64_t numel;
  int conv_c;      // CONV: input channels
};

struct Layout {
  size_t total = 0;
  size_t conv1_w = 0, conv1_b = 0, conv2_w = 0, conv2_b = 0;
  std::vector<EncLayer> enc;
  size_t lnp_g = 0, lnp_b = 0;
  size_t tok_emb = 0, pos_emb = 0;
  std::vector<DecLayer> dec;
  size_t xkv_w = 0, xkv_b = 0, lnf_g = 0, lnf_b = 0;
  size_t window = 0, cos_t = 0, sin_t = 0, fb = 0, fb_range = 0, sinus = 0;
  size_t self_kv = 0, cross_kv = 0;
  int64_t self_stride = 0, cross_stride = 0;   // elements per slot
  size_t pcm_stage = 0, pcm_ptrs = 0, pcm_n = 0, mel_raw = 0, mel_gmax = 0, mel_norm = 0,
         h1 = 0, x = 0, xn = 0, qkv = 0, vt = 0, att = 0, hid = 0, p_slots = 0;
  size_t vt_bytes = 0;
  size_t d_slots = 0, d_tokens = 0, d_pos = 0, d_h = 0, d_xn = 0, d_qkv = 0, d_att = 0,
         d_hid = 0, d_partial = 0, d_apart = 0, d_logits = 0, d_keys = 0, d_argmax = 0,
         d_flag = 0;
  size_t wstage = 0;
  int64_t wstage_floats = 0;
  std::vector<PackOp> pack;
  std::vector<std::pair<size_t, size_t>> zero_regions;   // (offset, bytes) zeroed before packing
};

struct TimedLaunch {
  int cls;
  hipEvent_t a, b;
  double flops, bytes;
  int64_t inst = -1;   // >= 0: one of several end events of a phase instance (max counts)
};

}  // namespace

struct asr_ctx {
  asr_model_cfg cfg{};
  int device = -1;
  int es = 4;                      // storage element size
  WaitQueue queue;
  std::unordered_map<int64_t, Request> waiting;   // submitted, not popped
  std::unordered_map<int64_t, Request> popped;    // popped, not prefilled
  std::vector<Slot> slots;
  // continuous batching (asr_serve_*): the engine owns the slots while on
  ServeEngine serve;
  bool serve_mode = false;
  bool serve_overlap = false;       // prefill on a second stream beside the decode rows
  int overlap_reserve = 0;          // CUs its persistent GEMMs leave to the decode rows
  hipStream_t pstream = nullptr;    // that stream (non-blocking, default priority)
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  // the encoder's clips split into enc_groups groups; groups after the first
  // run their layers on estream[] beside it (non-blocking, default priority)
  static constexpr int kEncGroups = 4;
  int enc_groups = 2;
  hipStream_t estream[kEncGroups - 1] = {};
  hipEvent_t ev_efork = nullptr, ev_ejoin[kEncGroups - 1] = {};
  std::unordered_map<int64_t, Request> serving;   // admitted, not finished (audio kept
                                                  // for a re-prefill after preemption)
  // decode steps replayed from HIP graphs, one per (rows, logits wanted),
  // captured on a private stream at the second step of that shape
  bool decode_graphs = true;
  hipStream_t cap_stream = nullptr;
  std::unordered_map<int32_t, hipGraphExec_t> dgraph;
  std::unordered_map<int32_t, int32_t> dshape_seen;
  Layout L;
  bool bound = false, loaded = false;
  char* base = nullptr;
  size_t bytes = 0;
  hipStream_t stream = nullptr;
  // timing
  int32_t timing = 0;   // bit mask over asr_kernel_class
  std::vector<hipEvent_t> ev_pool;
  size_t ev_used = 0;
  int64_t next_inst = 0;
  std::vector<TimedLaunch> pending;
  double t_ms[ASR_K_COUNT] = {}, t_flops[ASR_K_COUNT] = {}, t_bytes[ASR_K_COUNT] = {};
  int64_t t_n[ASR_K_COUNT] = {};

  template <typename T = char>
  T* at(size_t off) {
    return (T*)(base + off);
  }
  bool bf16() const { return cfg.dtype == ASR_BF16; }
};

namespace {

// ---------------------------------------------------------------------------
// Workspace plan
// ---------------------------------------------------------------------------
struct Bump {
  size_t off = 0;
  size_t take(size_t bytes) {
    off = (off + 255) / 256 * 256;
    size_t r = off;
    off += bytes;
    return r;
  }
};

void plan(asr_ctx* c) {
  const asr_model_cfg& g = c->cfg;
  const size_t es = c->es, f4 = 4;
  const int64_t d = g.d_model, F = g.d_ffn, M = g.n_mels, H = g.n_head;
  Layout& L = c->L;
  L = Layout();
  Bump b;
  int64_t max_param = 0;
  auto addp = [&](PackOp::Kind k, size_t dst, int64_t numel, int conv_c = 0) {
    L.pack.push_back({k, dst, numel, conv_c});
    max_param = std::max(max_param, numel);
  };
  if (g.n_enc > 0) {
    L.conv1_w = b.take(d * 3 * M * es);
    L.conv1_b = b.take(d * f4);
    L.conv2_w = b.take(d * 3 * d * es);
    L.conv2_b = b.take(d * f4);
    addp(PackOp::CONV, L.conv1_w, d * M * 3, (int)M);
    addp(PackOp::F32, L.conv1_b, d);
    addp(PackOp::CONV, L.conv2_w, d * d * 3, (int)d);
    addp(PackOp::F32, L.conv2_b, d);
    for (int l = 0; l < g.n_enc; ++l) {
      EncLayer e;
      e.ln1_g = b.take(d * f4); e.ln1_b = b.take(d * f4);
      e.qkv_w = b.take(3 * d * d * es); e.qkv_b = b.take(3 * d * f4);
      e.o_w = b.take(d * d * es); e.o_b = b.take(d * f4);
      e.ln2_g = b.take(d * f4); e.ln2_b = b.take(d * f4);
      e.fc1_w = b.take(F * d * es); e.fc1_b = b.take(F * f4);
      e.fc2_w = b.take(d * F * es); e.fc2_b = b.take(d * f4);
      L.enc.push_back(e);
      addp(PackOp::F32, e.ln1_g, d);
      addp(PackOp::F32, e.ln1_b, d);
      addp(PackOp::STORE, e.qkv_w, d * d);                     // q.w
      addp(PackOp::F32, e.qkv_b, d);                           // q.b
      addp(PackOp::STORE, e.qkv_w + d * d * es, d * d);        // k.w
      addp(PackOp::STORE, e.qkv_w + 2 * d * d * es, d * d);    // v.w
      addp(PackOp::F32, e.qkv_b + 2 * d * f4, d);              // v.b
      addp(PackOp::STORE, e.o_w, d * d);
      addp(PackOp::F32, e.o_b, d);
      addp(PackOp::F32, e.ln2_g, d);
      addp(PackOp::F32, e.ln2_b, d);
      addp(PackOp::STORE, e.fc1_w, F * d);
      addp(PackOp::F32, e.fc1_b, F);
      addp(PackOp::STORE, e.fc2_w, d * F);
      addp(PackOp::F32, e.fc2_b, d);
      L.zero_regions.push_back({e.qkv_b + d * f4, d * f4});     // k has no bias
    }
    L.lnp_g = b.take(d * f4);
    L.lnp_b = b.take(d * f4);
    addp(PackOp::F32, L.lnp_g, d);
    addp(PackOp::F32, L.lnp_b, d);
  }
  if (g.n_dec > 0) {
    const int64_t V = g.vocab;
    L.tok_emb = b.take(V * d * es);
    L.pos_emb = b.take(kTextCtx * d * f4);
    L.xkv_w = b.take((int64_t)g.n_dec * 2 * d * d * es);
    L.xkv_b = b.take((int64_t)g.n_dec * 2 * d * f4);
    addp(PackOp::STORE, L.tok_emb, V * d);
    addp(PackOp::F32, L.pos_emb, kTextCtx * d);
    for (int l = 0; l < g.n_dec; ++l) {
      DecLayer e;
      e.ln1_g = b.take(d * f4); e.ln1_b = b.take(d * f4);
      e.qkv_w = b.take(3 * d * d * es); e.qkv_b = b.take(3 * d * f4);
      e.o_w = b.take(d * d * es); e.o_b = b.take(d * f4);
      e.lnx_g = b.take(d * f4); e.lnx_b = b.take(d * f4);
      e.xq_w = b.take(d * d * es); e.xq_b = b.take(d * f4);
      e.xo_w = b.take(d * d * es); e.xo_b = b.take(d * f4);
      e.ln2_g = b.take(d * f4); e.ln2_b = b.take(d * f4);
      e.fc1_w = b.take(F * d * es); e.fc1_b = b.take(F * f4);
      e.fc2_w = b.take(d * F * es); e.fc2_b = b.take(d * f4);
      L.dec.push_back(e);
      size_t xk = L.xkv_w + (size_t)l * 2 * d * d * es, xb = L.xkv_b + (size_t)l * 2 * d * f4;
      addp(PackOp::F32, e.ln1_g, d);
      addp(PackOp::F32, e.ln1_b, d);
      addp(PackOp::STORE, e.qkv_w, d * d);
      addp(PackOp::F32, e.qkv_b, d);
      addp(PackOp::STORE, e.qkv_w + d * d * es, d * d);
      addp(PackOp::STORE, e.qkv_w + 2 * d * d * es, d * d);
      addp(PackOp::F32, e.qkv_b + 2 * d * f4, d);
      addp(PackOp::STORE, e.o_w, d * d);
      addp(PackOp::F32, e.o_b, d);
      addp(PackOp::F32, e.lnx_g, d);
      addp(PackOp::F32, e.lnx_b, d);
      addp(PackOp::STORE, e.xq_w, d * d);
      addp(PackOp::F32, e.xq_b, d);
      addp(PackOp::STORE, xk, d * d);                           // xk.w
      addp(PackOp::STORE, xk + d * d * es, d * d);              // xv.w
      addp(PackOp::F32, xb + d * f4, d);                        // xv.b
      addp(PackOp::STORE, e.xo_w, d * d);
      addp(PackOp::F32, e.xo_b, d);
      addp(PackOp::F32, e.ln2_g, d);
      addp(PackOp::F32, e.ln2_b, d);
      addp(PackOp::STORE, e.fc1_w, F * d);
      addp(PackOp::F32, e.fc1_b, F);
      addp(PackOp::STORE, e.fc2_w, d * F);
      addp(PackOp::F32, e.fc2_b, d);
      L.zero_regions.push_back({e.qkv_b + d * f4, d * f4});
      L.zero_regions.push_back({xb, d * f4});                   // cross k has no bias
    }
    L.lnf_g = b.take(d * f4);
    L.lnf_b = b.take(d * f4);
    addp(PackOp::F32, L.lnf_g, d);
    addp(PackOp::F32, L.lnf_b, d);
  }
  // constant tables
  L.window = b.take(kNFFT * f4);
  L.cos_t = b.take(kNFFT * f4);
  L.sin_t = b.take(kNFFT * f4);
  L.fb = b.take(2 * kBins * f4);   // packed: at most two filters per bin
  L.fb_range = b.take(M * 3 * 4);
  L.sinus = b.take((int64_t)kCtx * d * f4);
  // per-slot caches [slot][n_dec][2][H][ctx][64]
  const int64_t S = g.max_slots;
  L.self_stride = (int64_t)g.n_dec * 2 * H * kTextCtx * kHeadDim;
  L.cross_stride = (int64_t)g.n_dec * 2 * H * kCtx * kHeadDim;
  L.self_kv = b.take(S * L.self_stride * es);
  L.cross_kv = b.take(S * L.cross_stride * es);
  // prefill scratch
  const int64_t P = std::max(1, g.max_prefill), R = P * kCtx;
  L.pcm_stage = b.take(P * kSamples30s * f4);
  L.pcm_ptrs = b.take(P * 8);
  L.pcm_n = b.take(P * 8);
  L.mel_raw = b.take(P * kFrames * M * f4);
  L.mel_gmax = b.take(P * kMelGroups * 4);
  L.mel_norm = b.take(P * (kFrames + 2) * M * std::max<size_t>(es, f4));
  L.h1 = b.take(P * (kFrames + 1) * d * es);
  L.x = b.take(R * d * f4);
  L.xn = b.take(R * d * es);
  L.qkv = b.take(R * 3 * d * es);
  // per-head transposed V of the bf16 encoder attention, positions padded to
  // kVtLd with zeros (written once at bind, never touched by the kernels)
  L.vt_bytes = c->cfg.dtype == ASR_BF16 ? (size_t)P * H * kHeadDim * kVtLd * es : 0;
  L.vt = b.take(L.vt_bytes);
  L.att = b.take(R * d * es);
  L.hid = b.take(R * F * es);
  L.p_slots = b.take(P * 4);
  // decode scratch
  const int64_t D = std::max(1, g.max_decode);
  const int64_t Nmax = std::max<int64_t>(3 * d, F);
  L.d_slots = b.take(D * 4);
  L.d_tokens = b.take(D * 4);
  L.d_pos = b.take(D * 4);
  L.d_h = b.take(D * d * f4);
  L.d_xn = b.take(D * std::max<int64_t>(d, F) * es);
  L.d_qkv = b.take(D * 3 * d * es);
  L.d_att = b.take(D * d * es);
  L.d_hid = b.take(D * F * es);
  // partial sums of the decode products: the bf16 path splits the K range of
  // the products whose output feeds a residual LayerNorm or the cross
  // attention (N = d); the fp32 path holds one slice of any product
  {
    int64_t most = D * std::max<int64_t>(3 * d, F);
    if (c->cfg.dtype == ASR_BF16)
      most = std::max<int64_t>(
          most, std::max<int64_t>(D * d * std::max(dgemm_splits((int)d, (int)d),
                                                   dgemm_splits((int)d, (int)F)),
                                  D * 3 * d * dgemm_splits((int)(3 * d), (int)d)));
    L.d_partial = b.take(most * f4);
  }
  L.d_apart = b.take((int64_t)decode_attn_part_floats((int)D, g.n_head) * f4);
  L.d_logits = b.take(D * (int64_t)std::max(1, g.vocab) * f4);
  L.d_keys = b.take(D * (int64_t)vocab_tiles(std::max(1, g.vocab)) * 8);
  L.d_argmax = b.take(D * 4);
  L.d_flag = b.take(256);
  // staging for weight upload and debug read-back
  int64_t stage = max_param;
  stage = std::max<int64_t>(stage, P * kFrames * M);               // debug logmel
  stage = std::max<int64_t>(stage, P * (int64_t)kCtx * d);         // debug encode
  stage = std::max<int64_t>(stage, std::max(L.self_stride, L.cross_stride));
  L.wstage_floats = stage;
  L.wstage = b.take(stage * f4);
  L.total = (b.off + 255) / 256 * 256;
}

// ---------------------------------------------------------------------------
// Constant tables (computed here in double, stored as float)
// ---------------------------------------------------------------------------
double slaney_mel(double f) {
  const double f_sp = 200.0 / 3.0, min_log_hz = 1000.0, min_log_mel = 15.0;
  const double logstep = std::log(6.4) / 27.0;
  return f < min_log_hz ? f / f_sp : min_log_mel + std::log(f / min_log_hz) / logstep;
}
double slaney_hz(double m) {
  const double f_sp = 200.0 / 3.0, min_log_hz = 1000.0, min_log_mel = 15.0;
  const double logstep = std::log(6.4) / 27.0;
  return m < min_log_mel ? m * f_sp : min_log_hz * std::exp(logstep * (m - min_log_mel));
}

// Window, twiddles, mel filterbank (Slaney scale, area-normalised triangles
// over the 201 bins) packed as each filter's nonzero bin range, filter after
// filter, with [first bin, bin count, offset into the packed weights] per
// filter (at most 2 x 201 weights: a bin lies under at most two triangles).
struct HostMelTables {
  std::vector<float> win, ct, st, fb;
  std::vector<int32_t> rng;
};

HostMelTables host_mel_tables(int M) {
  HostMelTables t;
  t.win.resize(kNFFT);
  t.ct.resize(kNFFT);
  t.st.resize(kNFFT);
  for (int i = 0; i < kNFFT; ++i) {
    double a = 2.0 * M_PI * i / kNFFT;
    t.win[i] = (float)(0.5 - 0.5 * std::cos(a));
    t.ct[i] = (float)std::cos(a);
    t.st[i] = (float)std::sin(a);
  }
  std::vector<float> dense((size_t)M * kBins, 0.f);
  t.rng.assign((size_t)M * 3, 0);
  std::vector<double> edge(M + 2);
  double mlo = slaney_mel(0.0), mhi = slaney_mel(kSampleRate / 2.0);
  for (int i = 0; i < M + 2; ++i) edge[i] = slaney_hz(mlo + (mhi - mlo) * i / (M + 1));
  for (int m = 0; m < M; ++m) {
    int first = -1, last = -1;
    double norm = 2.0 / (edge[m + 2] - edge[m]);
    for (int k = 0; k < kBins; ++k) {
      double f = (double)k * kSampleRate / kNFFT;
      double up = (f - edge[m]) / (edge[m + 1] - edge[m]);
      double down = (edge[m + 2] - f) / (edge[m + 2] - edge[m + 1]);
      double w = std::max(0.0, std::min(up, down)) * norm;
      dense[(size_t)m * kBins + k] = (float)w;
      if (w > 0) {
        if (first < 0) first = k;
        last = k;
      }
    }
    t.rng[3 * m] = first < 0 ? 0 : first;
    t.rng[3 * m + 1] = first < 0 ? 0 : last - first + 1;
  }
  // packed nonzero range of every filter, filter after filter
  for (int m = 0; m < M; ++m) {
    t.rng[3 * m + 2] = (int32_t)t.fb.size();
    for (int i = 0; i < t.rng[3 * m + 1]; ++i)
      t.fb.push_back(dense[(size_t)m * kBins + t.rng[3 * m] + i]);
  }
  return t;
}

asr_status upload_tables(asr_ctx* c) {
  const int M = c->cfg.n_mels, d = c->cfg.d_model;
  const HostMelTables mt = host_mel_tables(M);
  // the kernel stages the packed weights in LDS sized for two per bin (every
  // bin lies in at most two triangular filters)
  if (mt.fb.size() > 2 * kBins) return fail(ASR_EINVAL, "packed filterbank larger than two weights per bin");
  const std::vector<float>&win = mt.win, &ct = mt.ct, &st = mt.st, &fb = mt.fb;
  const std::vector<int32_t>& rng = mt.rng;
  std::vector<float> sin_tab((size_t)kCtx * d);
  const int half = d / 2;
  const double inc = std::log(10000.0) / (half - 1);
  for (int t = 0; t < kCtx; ++t)
    for (int j = 0; j < half; ++j) {
      double a = t * std::exp(-inc * j);
      sin_tab[(size_t)t * d + j] = (float)std::sin(a);
      sin_tab[(size_t)t * d + half + j] = (float)std::cos(a);
    }
  hipStream_t s = c->stream;
  HIPCHK(hipMemcpyAsync(c->at(c->L.window), win.data(), kNFFT * 4, hipMemcpyHostToDevice, s));
  HIPCHK(hipMemcpyAsync(c->at(c->L.cos_t), ct.data(), kNFFT * 4, hipMemcpyHostToDevice, s));
  HIPCHK(hipMemcpyAsync(c->at(c->L.sin_t), st.data(), kNFFT * 4, hipMemcpyHostToDevice, s));
  HIPCHK(hipMemcpyAsync(c->at(c->L.fb), fb.data(), fb.size() * 4, hipMemcpyHostToDevice, s));
  HIPCHK(hipMemcpyAsync(c->at(c->L.fb_range), rng.data(), rng.size() * 4, hipMemcpyHostToDevice, s));
  HIPCHK(hipMemcpyAsync(c->at(c->L.sinus), sin_tab.data(), sin_tab.size() * 4,
                        hipMemcpyHostToDevice, s));
  if (c->L.vt_bytes) fill_u32(c->at<uint32_t>(c->L.vt), 0u, (int64_t)(c->L.vt_bytes / 4), s);
  HIPCHK(hipStreamSynchronize(s));
  return ASR_OK;
}

// ---------------------------------------------------------------------------
// Timing
// ---------------------------------------------------------------------------
hipEvent_t next_event(asr_ctx* c) {
  if (c->ev_used == c->ev_pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    c->ev_pool.push_back(e);
  }
  return c->ev_pool[c->ev_used++];
}

template <class F>
void timed(asr_ctx* c, int cls, double flops, double bytes, F&& f) {
  if (!(c->timing >> cls & 1)) {
    f();
    return;
  }
  hipEvent_t a = next_event(c), b = next_event(c);
  if (!a || !b) {
    f();
    return;
  }
  (void)hipEventRecord(a, c->stream);
  f();
  (void)hipEventRecord(b, c->stream);
  c->pending.push_back({cls, a, b, flops, bytes});
}

// Event pair around a whole phase of a step (recorded only when timing is on).
struct PhaseMark {
  asr_ctx* c;
  int cls;
  hipEvent_t a = nullptr;
  PhaseMark(asr_ctx* c_, int cls_) : c(c_), cls(cls_) {
    if (c->timing >> cls & 1) {
      a = next_event(c);
      if (a) (void)hipEventRecord(a, c->stream);
    }
  }
  void end() {
    if (!a) return;
    hipEvent_t b = next_event(c);
    if (!b) return;
    (void)hipEventRecord(b, c->stream);
    c->pending.push_back({cls, a, b, 0.0, 0.0});
    a = nullptr;
  }
};

asr_status collect_timing(asr_ctx* c) {
  if (c->pending.empty()) return ASR_OK;
  HIPCHK(hipDeviceSynchronize());
  std::unordered_map<int64_t, std::pair<int, float>> inst_ms;   // instance -> (class, max ms)
  for (auto& p : c->pending) {
    float ms = 0.f;
    HIPCHK(hipEventElapsedTime(&ms, p.a, p.b));
    if (p.inst >= 0) {
      auto it = inst_ms.find(p.inst);
      if (it == inst_ms.end())
        inst_ms[p.inst] = {p.cls, ms};
      else
        it->second.second = std::max(it->second.second, ms);
      continue;
    }
    c->t_ms[p.cls] += ms;
    c->t_n[p.cls] += 1;
    c->t_flops[p.cls] += p.flops;
    c->t_bytes[p.cls] += p.bytes;
  }
  for (auto& kv : inst_ms) {
    c->t_ms[kv.second.first] += kv.second.second;
    c->t_n[kv.second.first] += 1;
  }
  c->pending.clear();
  c->ev_used = 0;
  return ASR_OK;
}

// ---------------------------------------------------------------------------
// Encoder (prefill) pipeline
// ---------------------------------------------------------------------------
// Uploads the clips' sample pointers; host clips are first copied into the
// staging area.  Returns the number of clips prepared.
asr_status stage_pcm(asr_ctx* c, const float* const* pcm, const int64_t* n_samples, int n,
                     bool on_device) {
  std::vector<const float*> ptrs(n);
  std::vector<int64_t> ns(n);
  for (int i = 0; i < n; ++i) {
    if (n_samples[i] < 0 || n_samples[i] > kSamples30s)
      return fail(ASR_EINVAL, "n_samples out of [0, 480000]");
    ns[i] = n_samples[i];
    if (on_device) {
      ptrs[i] = pcm[i];
    } else {
      float* dst = c->at<float>(c->L.pcm_stage) + (size_t)i * kSamples30s;
      if (ns[i] > 0)
        HIPCHK(hipMemcpyAsync(dst, pcm[i], ns[i] * 4, hipMemcpyHostToDevice, c->stream));
      ptrs[i] = dst;
    }
    if (ns[i] > 0 && ptrs[i] == nullptr) return fail(ASR_EINVAL, "NULL pcm");
  }
  HIPCHK(hipMemcpyAsync(c->at(c->L.pcm_ptrs), ptrs.data(), n * 8, hipMemcpyHostToDevice, c->stream));
  HIPCHK(hipMemcpyAsync(c->at(c->L.pcm_n), ns.data(), n * 8, hipMemcpyHostToDevice, c->stream));
  return ASR_OK;
}

asr_status run_mel(asr_ctx* c, int n) {
  const int M = c->cfg.n_mels;
  MelTables t{c->at<float>(c->L.window), c->at<float>(c->L.cos_t), c->at<float>(c->L.sin_t),
              c->at<float>(c->L.fb), c->at<int32_t>(c->L.fb_range)};
  double bytes = 0;   // PCM read once, features written once (float32)
  bytes = (double)n * kSamples30s * 4 + (double)n * kFrames * M * 4;
  timed(c, ASR_K_MEL, (double)n * kFrames * kBins * kNFFT * 4.0, bytes, [&] {
    log_mel(c->at<const float* const>(c->L.pcm_ptrs), c->at<int64_t>(c->L.pcm_n), n, M, t,
            c->at<float>(c->L.mel_raw), c->at<float>(c->L.mel_gmax), c->stream);
  });
  CHECK_LAUNCH();
  return ASR_OK;
}

template <typename T>
void gemm_any(asr_ctx* c, const AView& a, size_t w_off, int M, int N, int K, const Epilogue& e) {
  double flops = 2.0 * M * N * K;
  // operands read once, result written once (the second convolution writes
  // the float32 stream)
  double out_bytes = (double)M * N * c->es;
  if (e.kind == EPI_CONV2) out_bytes = (double)M * N * 4;
  double bytes = (double)M * K * c->es + (double)N * K * c->es + out_bytes;
  timed(c, e.kind == EPI_XKV ? ASR_K_XKV : ASR_K_GEMM, flops, bytes, [&] {
    if (c->bf16())
      gemm_bf16(a, c->at<bf16_t>(w_off), M, N, K, e, c->stream);
    else
      gemm_f32(a, c->at<float>(w_off), M, N, K, e, c->stream);
  });
}

template <typename T>
void ln_any(asr_ctx* c, const float* x, int rows, size_t g, size_t b, T* out) {
  const int d = c->cfg.d_model;
  timed(c, ASR_K_LN, 8.0 * rows * d, (double)rows * d * (4 + c->es), [&] {
    layer_norm<T>(x, rows, d, c->at<float>(g), c->at<float>(b), out, c->stream);
  });
}

// The residual adds of a block fused with the LayerNorm that follows them
// (branch rows ldy elements apart): with y2, x = (x + y1) + y2 is stored and
// normalised; without, LayerNorm(x + y1) is formed and x is left as it was.
template <typename T>
void res_ln_any(asr_ctx* c, float* x, const T* y1, const T* y2, int64_t ldy, int rows, size_t g,
                size_t b, T* out) {
  const int d = c->cfg.d_model;
  const double bytes = y2 ? (double)rows * d * (8 + 3 * c->es) : (double)rows * d * (4 + 2 * c->es);
  timed(c, ASR_K_LN, 9.0 * rows * d, bytes, [&] {
    residual_layer_norm<T>(x, y1, y2, ldy, y2 != nullptr, rows, d, c->at<float>(g),
                           c->at<float>(b), out, c->stream);
  });
}

template <typename T>
asr_status cross_kv(asr_ctx* c, const void* E, int n, int slot0);

// mel -> stem -> encoder layers -> ln_post (-> with xkv, the cross K/V of
// every decoder layer into the slots in L.p_slots); E (storage type) ends in
// L.xn.
template <typename T>
asr_status encode_clips(asr_ctx* c, int n, bool xkv = false) {
  const asr_model_cfg& g = c->cfg;
  const int d = g.d_model, F = g.d_ffn, Mm = g.n_mels, H = g.n_head;
  const Layout& L = c->L;
  // the encoder phase (mel .. ln_post): starts here on the bound stream and
  // ends when the last clip group has its ln_post output
  hipEvent_t enc_a = nullptr;
  const int64_t enc_inst = c->next_inst++;
  if (c->timing >> ASR_K_ENCODE & 1) {
    enc_a = next_event(c);
    if (enc_a) (void)hipEventRecord(enc_a, c->stream);
  }
  auto enc_end = [&]() {
    if (!enc_a) return;
    hipEvent_t b = next_event(c);
    if (!b) return;
    (void)hipEventRecord(b, c->stream);
    TimedLaunch t{ASR_K_ENCODE, enc_a, b, 0.0, 0.0};
    t.inst = enc_inst;
    c->pending.push_back(t);
  };
  asr_status st = run_mel(c, n);
  if (st != ASR_OK) return st;
  timed(c, ASR_K_MEL, 0.0, (double)n * kFrames * Mm * (4 + c->es), [&] {
    mel_normalize<T>(c->at<float>(L.mel_raw), c->at<float>(L.mel_gmax), n, Mm,
                     c->at<T>(L.mel_norm), 1, c->stream);
  });
  float* x_all = c->at<float>(L.x);
  T* xn_all = c->at<T>(L.xn);
  T* qkv_all = c->at<T>(L.qkv);
  T* att_all = c->at<T>(L.att);
  T* hid_all = c->at<T>(L.hid);
  // The clips split into groups (two by default) whose layer chains run on
  // their own streams: while one group's memory-bound LayerNorm or the last
  // partial round of a persistent GEMM runs, another group's kernels fill the
  // idle CUs.  The groups own disjoint rows of every buffer.
  const int G = std::max(1, std::min(n, c->enc_groups));
  hipStream_t main_stream = c->stream;
  if (G > 1) {
    if (!c->ev_efork) {
      HIPCHK(hipEventCreateWithFlags(&c->ev_efork, hipEventDisableTiming));
      for (int i = 0; i < asr_ctx::kEncGroups - 1; ++i) {
        HIPCHK(hipStreamCreateWithFlags(&c->estream[i], hipStreamNonBlocking));
        HIPCHK(hipEventCreateWithFlags(&c->ev_ejoin[i], hipEventDisableTiming));
      }
    }
    HIPCHK(hipEventRecord(c->ev_efork, main_stream));
    for (int i = 0; i < G - 1; ++i) HIPCHK(hipStreamWaitEvent(c->estream[i], c->ev_efork, 0));
  }
  int clip0[asr_ctx::kEncGroups], nclip[asr_ctx::kEncGroups];
  for (int i = 0; i < G; ++i) {
    clip0[i] = n * i / G;
    nclip[i] = n * (i + 1) / G - clip0[i];
  }
  for (int l = 0; l <= g.n_enc; ++l) {
    for (int grp = 0; grp < G; ++grp) {
      c->stream = grp == 0 ? main_stream : c->estream[grp - 1];
      const int ng = nclip[grp], R = ng * kCtx;
      const int64_t r0 = (int64_t)clip0[grp] * kCtx;
      float* x = x_all + r0 * d;
      T* xn = xn_all + r0 * d;
      T* qkv = qkv_all + r0 * 3 * d;
      T* att = att_all + r0 * d;
      T* hid = hid_all + r0 * F;
      // The residual branches (attention out-projection, FC2) are written in
      // the storage type to ya and yf, which borrow the group's QKV rows
      // (dead once attention has run; rows 3d apart), and are added into the
      // float32 stream by the LayerNorm kernels that follow, as a model
      // stored in bf16 adds its bf16 branch outputs to the residual.  The
      // first LayerNorm normalises x + ya without storing it; the second
      // stores x = (x + ya) + yf (the same sums, one write of x per layer).
      T* ya = qkv;
      T* yf = qkv + d;
      if (l == 0) {
        // conv1: rows t of clip g read padded mel rows t .. t+2 (positions t-1 .. t+1)
        {
          AView a{c->at<T>(L.mel_norm) + (int64_t)clip0[grp] * (kFrames + 2) * Mm, Mm,
                  (int64_t)(kFrames + 2) * Mm, kFrames};
          Epilogue e{};
          e.kind = EPI_CONV1;
          e.out = c->at<T>(L.h1) + (int64_t)clip0[grp] * (kFrames + 1) * d;
          e.bias = c->at<float>(L.conv1_b);
          e.d_model = d;
          gemm_any<T>(c, a, L.conv1_w, ng * kFrames, d, 3 * Mm, e);
        }
        // conv2 (stride 2): output t reads h1 rows 2t .. 2t+2 (positions 2t-1 .. 2t+1)
        {
          AView a{c->at<T>(L.h1) + (int64_t)clip0[grp] * (kFrames + 1) * d, 2 * (int64_t)d,
                  (int64_t)(kFrames + 1) * d, kCtx};
          Epilogue e{};
          e.kind = EPI_CONV2;
          e.out = x;
          e.ldc = d;
          e.bias = c->at<float>(L.conv2_b);
          e.pos = c->at<float>(L.sinus);
          gemm_any<T>(c, a, L.conv2_w, R, d, 3 * d, e);
        }
        if (g.n_enc > 0) ln_any<T>(c, x, R, L.enc[0].ln1_g, L.enc[0].ln1_b, xn);
        continue;
      }
      const EncLayer& w = L.enc[l - 1];
      // xn holds LN_1(x) here
      {
        // bf16: q, k into the fused buffer and v transposed per head for the
        // flash-attention kernel; fp32: plain [R][3d]
        AView a{xn, d, 0, R};
        Epilogue e{};
        e.kind = c->bf16() ? EPI_QKV : EPI_STORE;
        e.out = qkv;
        e.ldc = 3 * d;
        e.bias = c->at<float>(w.qkv_b);
        e.d_model = d;
        e.n_head = H;
        e.out2 = c->bf16() ? (void*)(c->at<T>(L.vt) + (int64_t)clip0[grp] * H * kHeadDim * kVtLd)
                           : nullptr;
        gemm_any<T>(c, a, w.qkv_w, R, 3 * d, d, e);
      }
      timed(c, ASR_K_ATTN, 4.0 * ng * H * (double)kCtx * kCtx * 64,
            (double)R * 4 * d * c->es, [&] {
              if (c->bf16())
                flash_attn_bf16((const bf16_t*)qkv,
                                c->at<bf16_t>(L.vt) + (int64_t)clip0[grp] * H * kHeadDim * kVtLd,
                                (bf16_t*)att, ng, H, c->stream);
              else
                flash_attn_f32((const float*)qkv, (float*)att, ng, H, c->stream);
            });
      {
        AView a{att, d, 0, R};
        Epilogue e{};
        e.kind = EPI_STORE;
        e.out = ya;
        e.ldc = 3 * d;
        e.bias = c->at<float>(w.o_b);
        gemm_any<T>(c, a, w.o_w, R, d, d, e);
      }
      res_ln_any<T>(c, x, ya, nullptr, 3 * d, R, w.ln2_g, w.ln2_b, xn);
      {
        AView a{xn, d, 0, R};
        Epilogue e{};
        e.kind = EPI_GELU;
        e.out = hid;
        e.ldc = F;
        e.bias = c->at<float>(w.fc1_b);
        gemm_any<T>(c, a, w.fc1_w, R, F, d, e);
      }
      {
        AView a{hid, F, 0, R};
        Epilogue e{};
        e.kind = EPI_STORE;
        e.out = yf;
        e.ldc = 3 * d;
        e.bias = c->at<float>(w.fc2_b);
        gemm_any<T>(c, a, w.fc2_w, R, d, F, e);
      }
      // the next LayerNorm: the next layer's LN_1, or ln_post after the last layer
      const bool last = l == g.n_enc;
      res_ln_any<T>(c, x, ya, yf, 3 * d, R, last ? L.lnp_g : L.enc[l].ln1_g,
                    last ? L.lnp_b : L.enc[l].ln1_b, xn);
      if (last) enc_end();
    }
  }
  c->stream = main_stream;
  for (int i = 0; i < G - 1; ++i) {
    HIPCHK(hipEventRecord(c->ev_ejoin[i], c->estream[i]));
    HIPCHK(hipStreamWaitEvent(main_stream, c->ev_ejoin[i], 0));
  }
  if (g.n_enc == 0) {
    ln_any<T>(c, x_all, n * kCtx, L.lnp_g, L.lnp_b, xn_all);
    enc_end();
  }
  // the cross K/V of all clips as one product, after the groups have joined
  // (a persistent GEMM fills every CU by itself, so splitting it by group
  // gains nothing, and the encoder phase then ends where the product starts)
  if (xkv) {
    const asr_status st2 = cross_kv<T>(c, xn_all, n, 0);
    if (st2 != ASR_OK) return st2;
  }
  CHECK_LAUNCH();
  return ASR_OK;
}

// Projects E (storage type, [n][1500][d] at `E`) into the cross caches of
// the slots listed in device array L.p_slots from entry slot0 on.
template <typename T>
asr_status cross_kv(asr_ctx* c, const void* E, int n, int slot0) {
  const asr_model_cfg& g = c->cfg;
  const int d = g.d_model;
  AView a{E, d, 0, n * kCtx};
  Epilogue e{};
  e.kind = EPI_XKV;
  e.out = c->at(c->L.cross_kv);
  e.bias = c->at<float>(c->L.xkv_b);
  e.slots = c->at<int32_t>(c->L.p_slots) + slot0;
  e.slot_stride = c->L.cross_stride;
  e.d_model = d;
  e.n_head = g.n_head;
  gemm_any<T>(c, a, c->L.xkv_w, n * kCtx, g.n_dec * 2 * d, d, e);
  CHECK_LAUNCH();
  return ASR_OK;
}

// ---------------------------------------------------------------------------
// Decode pipeline (rows already uploaded to d_slots / d_tokens / d_pos)
// ---------------------------------------------------------------------------
// Decode product with its epilogue: out = (GELU)(x W^T + bias) in the
// storage type.  bf16: one kernel; fp32: the product, then the epilogue.
template <typename T>
void dgemm_out(asr_ctx* c, const T* x, size_t w_off, int D, int N, int K, size_t bias_off,
               bool gelu, T* out) {
  float* part = c->at<float>(c->L.d_partial);
  const double bytes = (double)N * K * c->es + (double)D * K * c->es + (double)D * N * c->es;
  timed(c, ASR_K_DGEMM, 2.0 * D * N * K, bytes, [&] {
    if (c->bf16()) {
      dgemm_bf16((const bf16_t*)x, c->at<bf16_t>(w_off), D, N, K, gelu ? DG_GELU : DG_BIAS,
                 c->at<float>(bias_off), out, c->stream);
    } else {
      dgemm_f32((const float*)x, c->at<float>(w_off), D, N, K, part, c->stream);
      dgemm_reduce<T>(part, 1, D, N, c->at<float>(bias_off), gelu ? 1 : 0, out, c->stream);
    }
  });
}

// Decode product left as float32 partial sums over K slices in d_partial
// (the consumer adds the slices and the bias); returns the slice count.
template <typename T>
int dgemm_part(asr_ctx* c, const T* x, size_t w_off, int D, int N, int K) {
  float* part = c->at<float>(c->L.d_partial);
  int splits = 1;
  const double bytes = (double)N * K * c->es + (double)D * K * c->es + (double)D * N * c->es;
  timed(c, ASR_K_DGEMM, 2.0 * D * N * K, bytes, [&] {
    if (c->bf16())
      splits = dgemm_bf16((const bf16_t*)x, c->at<bf16_t>(w_off), D, N, K, DG_PARTIAL, nullptr,
                          part, c->stream);
    else
      dgemm_f32((const float*)x, c->at<float>(w_off), D, N, K, part, c->stream);
  });
  return splits;
}

// Residual product (N = d): h += bias + x W^T, then xn = LayerNorm(h) with
// (g, b) -- the product's K slices are added by the LayerNorm kernel.
template <typename T>
void dgemm_resid_ln(asr_ctx* c, const T* x, size_t w_off, int D, int K, size_t bias_off,
                    float* h, size_t g_off, size_t b_off, T* xn) {
  const int d = c->cfg.d_model;
  const int splits = dgemm_part<T>(c, x, w_off, D, d, K);
  timed(c, ASR_K_LN, 9.0 * D * d, (double)D * d * (4.0 * splits + 8 + c->es), [&] {
    reduce_resid_ln<T>(c->at<float>(c->L.d_partial), splits, D, d, c->at<float>(bias_off), h,
                       c->at<float>(g_off), c->at<float>(b_off), xn, c->stream);
  });
}

template <typename T>
asr_status decode_rows(asr_ctx* c, int D, const std::vector<int32_t>& pos_host, bool want_logits) {
  const asr_model_cfg& g = c->cfg;
  const int d = g.d_model, F = g.d_ffn, H = g.n_head, V = g.vocab;
  const Layout& L = c->L;
  float* h = c->at<float>(L.d_h);
  T* xn = c->at<T>(L.d_xn);
  T* qkv = c->at<T>(L.d_qkv);
  T* att = c->at<T>(L.d_att);
  T* hid = c->at<T>(L.d_hid);
  const int32_t* slots = c->at<int32_t>(L.d_slots);
  const int32_t* pos = c->at<int32_t>(L.d_pos);
  T* self_cache = c->at<T>(L.self_kv);
  T* cross_cache = c->at<T>(L.cross_kv);
  double self_keys = 0;
  for (int i = 0; i < D; ++i) self_keys += pos_host[i] + 1;

  timed(c, ASR_K_OTHER, 0.0, (double)D * d * (c->es + 8), [&] {
    embed<T>(c->at<T>(L.tok_emb), c->at<float>(L.pos_emb), c->at<int32_t>(L.d_tokens), pos, D, d,
             h, c->stream);
  });
  ln_any<T>(c, h, D, L.dec[0].ln1_g, L.dec[0].ln1_b, xn);
  for (int l = 0; l < g.n_dec; ++l) {
    const DecLayer& w = L.dec[l];
    // xn holds LN_attn(h) here; bf16: the QKV product stays in K-slice
    // partial sums that the self-attention kernel adds up with the bias
    int qkv_splits = 0;
    if (c->bf16())
      qkv_splits = dgemm_part<T>(c, xn, w.qkv_w, D, 3 * d, d);
    else
      dgemm_out<T>(c, xn, w.qkv_w, D, 3 * d, d, w.qkv_b, false, qkv);
    const int64_t self_off = (int64_t)l * 2 * H * kTextCtx * kHeadDim;
    timed(c, ASR_K_DATTN, 4.0 * self_keys * 64 * H, self_keys * 2 * 64 * H * c->es, [&] {
      decode_self_attn<T>(qkv, c->at<float>(L.d_partial), qkv_splits, c->at<float>(w.qkv_b),
                          self_cache, L.self_stride, self_off, slots, pos, D, H, att,
                          c->at<float>(L.d_apart), c->stream);
    });
    dgemm_resid_ln<T>(c, att, w.o_w, D, d, w.o_b, h, w.lnx_g, w.lnx_b, xn);
    const int q_splits = dgemm_part<T>(c, xn, w.xq_w, D, d, d);
    const int64_t cross_off = (int64_t)l * 2 * H * kCtx * kHeadDim;
    timed(c, ASR_K_DATTN, 4.0 * D * H * (double)kCtx * 64, (double)D * H * kCtx * 2 * 64 * c->es,
          [&] {
            decode_cross_attn<T>(c->at<float>(L.d_partial), q_splits, c->at<float>(w.xq_b),
                                 cross_cache, L.cross_stride, cross_off, slots, D, H, att,
                                 c->at<float>(L.d_apart), c->stream);
          });
    dgemm_resid_ln<T>(c, att, w.xo_w, D, d, w.xo_b, h, w.ln2_g, w.ln2_b, xn);
    dgemm_out<T>(c, xn, w.fc1_w, D, F, d, w.fc1_b, true, hid);
    // the last residual of the layer also produces the next LayerNorm input
    const bool last = l + 1 == g.n_dec;
    dgemm_resid_ln<T>(c, hid, w.fc2_w, D, F, w.fc2_b, h, last ? L.lnf_g : L.dec[l + 1].ln1_g,
                      last ? L.lnf_b : L.dec[l + 1].ln1_b, xn);
  }
  const int nt = vocab_tiles(V);
  int32_t* flag = c->at<int32_t>(L.d_flag);
  fill_u32((uint32_t*)flag, 0u, 1, c->stream);
  timed(c, ASR_K_VOCAB, 2.0 * D * (double)V * d, (double)V * d * c->es + (double)D * d * c->es,
        [&] {
          if (c->bf16()) {
            vocab_argmax_bf16((const bf16_t*)xn, c->at<bf16_t>(L.tok_emb), D, V, d,
                              c->at<uint64_t>(L.d_keys), nt,
                              want_logits ? c->at<float>(L.d_logits) : nullptr, c->stream);
          } else {
            vocab_logits_f32((const float*)xn, c->at<float>(L.tok_emb), D, V, d,
                             c->at<float>(L.d_logits), c->stream);
            logits_argmax_keys(c->at<float>(L.d_logits), D, V, c->at<uint64_t>(L.d_keys), nt,
                               c->stream);
          }
          argmax_finish(c->at<uint64_t>(L.d_keys), D, nt, c->at<int32_t>(L.d_argmax), flag,
                        c->stream);
        });
  CHECK_LAUNCH();
  return ASR_OK;
}

asr_status need_gpu(const asr_ctx* c, bool need_loaded) {
  if (!c) return fail(ASR_EINVAL, "NULL context");
  if (c->device < 0) return fail(ASR_ENODEV, "queue-only context (device = -1)");
  if (!c->bound) return fail(ASR_ESTATE, "asr_bind has not been called");
  if (need_loaded && !c->loaded) return fail(ASR_ESTATE, "asr_load_weights has not been called");
  return ASR_OK;
}

int32_t steps_for(int64_t n_samples, int32_t max_tokens) {
  int64_t s = (27 * n_samples + 80000) / 160000;   // round-half-up of 2.7 tokens per second
  if (s < 1) s = 1;
  if (s > kTextCtx) s = kTextCtx;
  if (s > max_tokens) s = max_tokens;
  return (int32_t)s;
}

int free_slot(asr_ctx* c, const std::vector<int>& taken) {
  for (int s = 0; s < c->cfg.max_slots; ++s)
    if (!c->slots[s].occupied && std::find(taken.begin(), taken.end(), s) == taken.end())
      return s;
  return -1;
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

const char* asr_last_error(void) { return g_err.c_str(); }

asr_status asr_create(const asr_model_cfg* cfg, int32_t device, asr_ctx** out) {
  if (!cfg || !out) return fail(ASR_EINVAL, "NULL argument");
  const asr_model_cfg& g = *cfg;
  if (g.n_mels <= 0 || g.d_model <= 0 || g.n_head <= 0 || g.d_model != 64 * g.n_head)
    return fail(ASR_EINVAL, "d_model must equal 64 * n_head");
  if (g.n_mels % 8 != 0 || g.n_mels > 128)
    return fail(ASR_EINVAL, "n_mels must be a multiple of 8, at most 128");
  if (g.d_model > 2048) return fail(ASR_EINVAL, "d_model must be <= 2048");
  if (g.d_ffn <= 0 || g.d_ffn % 64 != 0) return fail(ASR_EINVAL, "d_ffn must be a multiple of 64");
  if (g.dtype == ASR_BF16 && (g.d_model % 128 != 0 || g.d_ffn % 128 != 0))
    return fail(ASR_EINVAL, "bf16 models need d_model and d_ffn multiples of 128");
  if (g.n_enc < 0 || g.n_dec < 0 || (g.n_enc == 0 && g.n_dec == 0))
    return fail(ASR_EINVAL, "need encoder or decoder layers");
  if (g.n_dec > 0 && g.vocab <= 0) return fail(ASR_EINVAL, "vocab must be positive");
  if (g.dtype != ASR_F32 && g.dtype != ASR_BF16) return fail(ASR_EINVAL, "dtype");
  if (g.max_slots < 0 || g.max_prefill < 0 || g.max_decode < 0 || g.max_queue <= 0 ||
      g.max_decode > std::max(g.max_slots, 0))
    return fail(ASR_EINVAL, "capacities (max_decode <= max_slots, max_queue > 0)");
  if (g.max_decode > 128) return fail(ASR_EINVAL, "max_decode must be <= 128");
  if (device < -1) return fail(ASR_EINVAL, "device");
  if (device >= 0) {
    int n = 0;
    hipError_t e = hipGetDeviceCount(&n);
    if (e != hipSuccess)
      return fail(ASR_ENODEV, std::string("hipGetDeviceCount: ") + hipGetErrorString(e));
    if (device >= n)
      return fail(ASR_ENODEV, "device " + std::to_string(device) + " of " + std::to_string(n));
  }
  asr_ctx* c = new asr_ctx();
  c->cfg = g;
  c->device = device;
  c->es = g.dtype == ASR_BF16 ? 2 : 4;
  c->slots.assign(std::max(g.max_slots, 0), Slot());
  c->queue.set_policy(WaitQueue::FCFS, 0, 0);
  plan(c);
  *out = c;
  return ASR_OK;
}

asr_status asr_destroy(asr_ctx* c) {
  if (!c) return ASR_OK;
  if (c->device >= 0) {
    (void)hipSetDevice(c->device);
    for (auto e : c->ev_pool) (void)hipEventDestroy(e);
    if (c->pstream) (void)hipStreamSynchronize(c->pstream);
    if (c->ev_fork) (void)hipEventDestroy(c->ev_fork);
    if (c->ev_join) (void)hipEventDestroy(c->ev_join);
    if (c->pstream) (void)hipStreamDestroy(c->pstream);
    for (int i = 0; i < asr_ctx::kEncGroups - 1; ++i) {
      if (c->estream[i]) (void)hipStreamSynchronize(c->estream[i]);
      if (c->ev_ejoin[i]) (void)hipEventDestroy(c->ev_ejoin[i]);
      if (c->estream[i]) (void)hipStreamDestroy(c->estream[i]);
    }
    if (c->ev_efork) (void)hipEventDestroy(c->ev_efork);
    for (auto& kv : c->dgraph) (void)hipGraphExecDestroy(kv.second);
    if (c->cap_stream) (void)hipStreamDestroy(c->cap_stream);
  }
  delete c;
  return ASR_OK;
}

asr_status asr_workspace_size(const asr_ctx* c, size_t* bytes) {
  if (!c || !bytes) return fail(ASR_EINVAL, "NULL argument");
  *bytes = c->L.total;
  return ASR_OK;
}

asr_status asr_bind(asr_ctx* c, void* dev_block, size_t bytes, void* stream) {
  if (!c) return fail(ASR_EINVAL, "NULL context");
  if (c->device < 0) return fail(ASR_ENODEV, "queue-only context (device = -1)");
  if (!dev_block || ((uintptr_t)dev_block & 255)) return fail(ASR_EINVAL, "block must be 256-byte aligned");
  if (bytes < c->L.total) return fail(ASR_ENOMEM, "bound block smaller than asr_workspace_size");
  HIPCHK(hipSetDevice(c->device));
  for (auto& kv : c->dgraph) (void)hipGraphExecDestroy(kv.second);
  c->dgraph.clear();
  c->dshape_seen.clear();
  c->base = (char*)dev_block;
  c->bytes = bytes;
  c->stream = (hipStream_t)stream;
  c->bound = true;
  c->loaded = false;
  return upload_tables(c);
}

asr_status asr_n_params(const asr_ctx* c, int32_t* n) {
  if (!c || !n) return fail(ASR_EINVAL, "NULL argument");
  *n = (int32_t)c->L.pack.size();
  return ASR_OK;
}

asr_status asr_param_numel(const asr_ctx* c, int32_t i, int64_t* numel) {
  if (!c || !numel) return fail(ASR_EINVAL, "NULL argument");
  if (i < 0 || i >= (int32_t)c->L.pack.size()) return fail(ASR_EINVAL, "parameter index");
  *numel = c->L.pack[i].numel;
  return ASR_OK;
}

asr_status asr_load_weights(asr_ctx* c, const float* const* tensors, int32_t n, int32_t on_device) {
  asr_status st = need_gpu(c, false);
  if (st != ASR_OK) return st;
  if (!tensors || n != (int32_t)c->L.pack.size()) return fail(ASR_EINVAL, "expected asr_n_params tensors");
  HIPCHK(hipSetDevice(c->device));
  hipStream_t s = c->stream;
  for (auto& z : c->L.zero_regions) fill_u32(c->at<uint32_t>(z.first), 0u, z.second / 4, s);
  float* stage = c->at<float>(c->L.wstage);
  for (int i = 0; i < n; ++i) {
    const PackOp& p = c->L.pack[i];
    if (!tensors[i]) return fail(ASR_EINVAL, "NULL tensor " + std::to_string(i));
    HIPCHK(hipMemcpyAsync(stage, tensors[i], p.numel * 4,
                          on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice, s));
    if (p.kind == PackOp::F32) {
      convert_from_f32<float>(stage, c->at<float>(p.dst), p.numel, s);
    } else if (p.kind == PackOp::STORE) {
      if (c->bf16())
        convert_from_f32<bf16_t>(stage, c->at<bf16_t>(p.dst), p.numel, s);
      else
        convert_from_f32<float>(stage, c->at<float>(p.dst), p.numel, s);
    } else {
      int dd = c->cfg.d_model;
      if (c->bf16())
        pack_conv<bf16_t>(stage, c->at<bf16_t>(p.dst), dd, p.conv_c, s);
      else
        pack_conv<float>(stage, c->at<float>(p.dst), dd, p.conv_c, s);
    }
    CHECK_LAUNCH();
    if (!on_device) HIPCHK(hipStreamSynchronize(s));   // staging reused by the next tensor
  }
  HIPCHK(hipStreamSynchronize(s));
  c->loaded = true;
  return ASR_OK;
}

asr_status asr_set_policy(asr_ctx* c, int32_t policy, int32_t kappa_num, int32_t kappa_den) {
  if (!c) return fail(ASR_EINVAL, "NULL context");
  if (policy < ASR_FCFS || policy > ASR_HRRN) return fail(ASR_EINVAL, "policy");
  if (kappa_den < 0 || (kappa_den > 0 && kappa_num <= 0))
    return fail(ASR_EINVAL, "kappa must be positive (or kappa_den = 0 for the duration key)");
  c->queue.set_policy(policy, kappa_num, kappa_den);
  return ASR_OK;
}

asr_status asr_submit(asr_ctx* c, int64_t id, const float* pcm, int64_t n_samples,
                      int32_t sample_rate, int64_t duration_us, int64_t arrival_us,
                      int32_t max_tokens, int32_t pcm_on_device) {
  if (!c) return fail(ASR_EINVAL, "NULL context");
  if (sample_rate != kSampleRate) return fail(ASR_EINVAL, "sample_rate must be 16000");
  if (n_samples < 0 || n_samples > kSamples30s)
    return fail(ASR_EINVAL, "n_samples must be in [0, 480000] (one 30-s segment)");
  if (n_samples == 0 && (pcm != nullptr || duration_us <= 0))
    return fail(ASR_EINVAL, "a request without samples needs pcm = NULL and duration_us > 0");
  if (max_tokens > kTextCtx) return fail(ASR_EINVAL, "max_tokens must be <= 448");
  if (c->queue.contains(id) || c->waiting.count(id) || c->popped.count(id) ||
      c->serving.count(id) || c->serve.has_result(id))
    return fail(ASR_EINVAL, "duplicate request id " + std::to_string(id));
  if ((int64_t)c->queue.size() >= c->cfg.max_queue) return fail(ASR_EFULL, "queue full");
  Request r;
  r.id = id;
  r.arrival_us = arrival_us;
  r.n_samples = n_samples;
  r.sample_rate = sample_rate;
  r.dur_us = duration_us > 0 ? duration_us : (n_samples * 1000000) / sample_rate;
  r.max_tokens = max_tokens > 0 ? max_tokens : kTextCtx;
  if (pcm) {
    r.has_audio = true;
    if (pcm_on_device)
      r.dev_pcm = pcm;
    else
      r.pcm.assign(pcm, pcm + n_samples);
  }
  QEntry e{id, r.arrival_us, r.n_samples, r.dur_us, r.sample_rate, r.max_tokens, 0};
  if (c->serve_mode) {
    const ServeConfig& sc = c->serve.config();
    if (sc.kv_capacity > 0 && (int64_t)sc.cross_tokens + c->serve.tokens_for(e) > sc.kv_capacity)
      return fail(ASR_EINVAL, "request can never fit the KV pool (cross share + its tokens)");
  }
  c->queue.push(e);
  c->waiting.emplace(id, std::move(r));
  return ASR_OK;
}

asr_status asr_rank(const asr_ctx* c, int64_t now_us, int64_t* out_ids, int32_t cap, int32_t* n_out) {
  if (!c || !n_out || (cap > 0 && !out_ids)) return fail(ASR_EINVAL, "NULL argument");
  std::vector<int64_t> ids = c->queue.rank(now_us);
  int32_t k = (int32_t)std::min<size_t>(ids.size(), (size_t)std::max(cap, 0));
  for (int32_t i = 0; i < k; ++i) out_ids[i] = ids[i];
  *n_out = k;
  return ASR_OK;
}

asr_status asr_pop_batch(asr_ctx* c, int64_t now_us, int32_t max_n, int64_t* out_ids, int32_t* n_out) {
  if (!c || !n_out || (max_n > 0 && !out_ids)) return fail(ASR_EINVAL, "NULL argument");
  if (c->serve_mode) return fail(ASR_ESTATE, "context is in continuous-batching mode (asr_serve_*)");
  std::vector<QEntry> got = c->queue.pop_batch(now_us, max_n);
  for (size_t i = 0; i < got.size(); ++i) {
    out_ids[i] = got[i].id;
    auto it = c->waiting.find(got[i].id);
    c->popped.emplace(got[i].id, std::move(it->second));
    c->waiting.erase(it);
  }
  *n_out = (int32_t)got.size();
  return ASR_OK;
}

asr_status asr_queue_len(const asr_ctx* c, int32_t* n) {
  if (!c || !n) return fail(ASR_EINVAL, "NULL argument");
  *n = (int32_t)c->queue.size();
  return ASR_OK;
}

asr_status asr_release_slot(asr_ctx* c, int32_t slot) {
  if (!c) return fail(ASR_EINVAL, "NULL context");
  if (c->serve_mode) return fail(ASR_ESTATE, "context is in continuous-batching mode (asr_serve_*)");
  if (slot < 0 || slot >= c->cfg.max_slots) return fail(ASR_ENOTFOUND, "no such slot");
  c->slots[slot] = Slot();
  return ASR_OK;
}

asr_status asr_slot_info(const asr_ctx* c, int32_t slot, int32_t* occupied, int64_t* id,
                         int32_t* position, int32_t* steps_left) {
  if (!c) return fail(ASR_EINVAL, "NULL context");
  if (slot < 0 || slot >= c->cfg.max_slots) return fail(ASR_ENOTFOUND, "no such slot");
  const Slot& s = c->slots[slot];
  if (occupied) *occupied = s.occupied;
  if (id) *id = s.id;
  if (position) *position = s.pos;
  if (steps_left) *steps_left = s.steps_left;
  return ASR_OK;
}

// ---------------------------------------------------------------------------
// Step execution shared by asr_step and asr_serve_step
// ---------------------------------------------------------------------------
}  // extern "C"

namespace {

// Host arrays a prefill's copies read; they must outlive the stream's sync.
struct PrefillStage {
  std::vector<const float*> ptrs;
  std::vector<int64_t> ns;
  std::vector<int32_t> slots;
};

// Prefill: audio of reqs[i] -> mel -> stem -> encoder -> cross K/V of slot
// slots[i], enqueued on c->stream (no synchronisation).
asr_status launch_prefill(asr_ctx* c, const std::vector<const Request*>& reqs,
                          const std::vector<int32_t>& slots_in, PrefillStage& stage) {
  const int P = (int)reqs.size();
  if (P == 0) return ASR_OK;
  hipStream_t s = c->stream;
  std::vector<const float*>& ptrs = stage.ptrs;
  std::vector<int64_t>& ns = stage.ns;
  std::vector<int32_t>& slots = stage.slots;
  ptrs.assign(P, nullptr);
  ns.assign(P, 0);
  slots = slots_in;
  bool any_host = false;
  for (int i = 0; i < P; ++i) {
    ns[i] = reqs[i]->n_samples;
    if (reqs[i]->dev_pcm) {
      ptrs[i] = reqs[i]->dev_pcm;
    } else {
      // host clips are uploaded into staging; every clip then reads device memory
      float* dst = c->at<float>(c->L.pcm_stage) + (size_t)i * kSamples30s;
      HIPCHK(hipMemcpyAsync(dst, reqs[i]->pcm.data(), ns[i] * 4, hipMemcpyHostToDevice, s));
      ptrs[i] = dst;
      any_host = true;
    }
  }
  HIPCHK(hipMemcpyAsync(c->at(c->L.pcm_ptrs), ptrs.data(), P * 8, hipMemcpyHostToDevice, s));
  HIPCHK(hipMemcpyAsync(c->at(c->L.pcm_n), ns.data(), P * 8, hipMemcpyHostToDevice, s));
  HIPCHK(hipMemcpyAsync(c->at(c->L.p_slots), slots.data(), P * 4, hipMemcpyHostToDevice, s));
  PhaseMark pm(c, ASR_K_PREFILL);
  const bool xkv = c->cfg.n_dec > 0;
  asr_status st = c->bf16() ? encode_clips<bf16_t>(c, P, xkv) : encode_clips<float>(c, P, xkv);
  if (st != ASR_OK) return st;
  pm.end();
  (void)any_host;
  return ASR_OK;
}

asr_status run_prefill(asr_ctx* c, const std::vector<const Request*>& reqs,
                       const std::vector<int32_t>& slots) {
  PrefillStage stage;
  asr_status st = launch_prefill(c, reqs, slots, stage);
  // the host arrays of the stage (and the pageable clips) must outlive the
  // copies that read them
  HIPCHK(hipStreamSynchronize(c->stream));
  return st;
}

// Enqueues the decode kernels of D rows on c->stream: directly, or by
// replaying the HIP graph of this shape.  Every argument of those kernels is
// a device pointer or a size fixed by (D, logits wanted) -- positions, slots
// and tokens are read from device memory -- so one graph serves every step of
// a shape.  A shape's first step runs directly (it also performs the
// kernels' one-time attribute set-up); the second is captured on a private
// stream and replayed from then on.  Per-launch timing always runs directly.
asr_status decode_launch(asr_ctx* c, int D, const std::vector<int32_t>& pos, bool want_logits) {
  auto direct = [&]() {
    return c->bf16() ? decode_rows<bf16_t>(c, D, pos, want_logits)
                     : decode_rows<float>(c, D, pos, want_logits);
  };
  const int32_t key = D * 2 + (want_logits ? 1 : 0);
  const bool per_launch_timing = (c->timing & ~((1 << ASR_K_PREFILL) | (1 << ASR_K_DECODE) |
                                                (1 << ASR_K_ENCODE))) != 0;
  if (!c->decode_graphs || per_launch_timing) return direct();
  auto it = c->dgraph.find(key);
  if (it == c->dgraph.end()) {
    if (c->dshape_seen[key]++ == 0) return direct();
    if (!c->cap_stream) HIPCHK(hipStreamCreateWithFlags(&c->cap_stream, hipStreamNonBlocking));
    hipStream_t bound = c->stream;
    c->stream = c->cap_stream;
    HIPCHK(hipStreamBeginCapture(c->cap_stream, hipStreamCaptureModeThreadLocal));
    asr_status st = direct();
    hipGraph_t g = nullptr;
    const hipError_t e = hipStreamEndCapture(c->cap_stream, &g);
    c->stream = bound;
    if (st != ASR_OK) {
      if (g) (void)hipGraphDestroy(g);
      return st;
    }
    if (e != hipSuccess) return fail(ASR_EDEVICE, std::string("hipStreamEndCapture: ") + hipGetErrorString(e));
    hipGraphExec_t ex = nullptr;
    const hipError_t e2 = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (e2 != hipSuccess) return fail(ASR_EDEVICE, std::string("hipGraphInstantiate: ") + hipGetErrorString(e2));
    it = c->dgraph.emplace(key, ex).first;
  }
  HIPCHK(hipGraphLaunch(it->second, c->stream));
  return ASR_OK;
}

// Decode rows (slot, token, position) -> argmax (and logits when asked).
// Returns EDEVICE after the copies when a NaN logit was flagged.
asr_status run_decode(asr_ctx* c, int D, const int32_t* slots, const int32_t* tokens,
                      const std::vector<int32_t>& pos, int32_t* argmax, float* logits) {
  if (D == 0) return ASR_OK;
  hipStream_t s = c->stream;
  HIPCHK(hipMemcpyAsync(c->at(c->L.d_slots), slots, D * 4, hipMemcpyHostToDevice, s));
  HIPCHK(hipMemcpyAsync(c->at(c->L.d_tokens), tokens, D * 4, hipMemcpyHostToDevice, s));
  HIPCHK(hipMemcpyAsync(c->at(c->L.d_pos), pos.data(), D * 4, hipMemcpyHostToDevice, s));
  PhaseMark pm(c, ASR_K_DECODE);
  asr_status st = decode_launch(c, D, pos, logits != nullptr);
  if (st != ASR_OK) return st;
  pm.end();
  int32_t flag = 0;
  HIPCHK(hipMemcpyAsync(argmax, c->at(c->L.d_argmax), D * 4, hipMemcpyDeviceToHost, s));
  HIPCHK(hipMemcpyAsync(&flag, c->at(c->L.d_flag), 4, hipMemcpyDeviceToHost, s));
  if (logits)
    HIPCHK(hipMemcpyAsync(logits, c->at(c->L.d_logits), (size_t)D * c->cfg.vocab * 4,
                          hipMemcpyDeviceToHost, s));
  HIPCHK(hipStreamSynchronize(s));
  if (flag) return fail(ASR_EDEVICE, "NaN logit");
  return ASR_OK;
}

}  // namespace

extern "C" {

asr_status asr_step(asr_ctx* c, const asr_step_in* in, asr_step_out* out) {
  asr_status st = need_gpu(c, true);
  if (st != ASR_OK) return st;
  if (!in || !out) return fail(ASR_EINVAL, "NULL argument");
  if (c->serve_mode) return fail(ASR_ESTATE, "context is in continuous-batching mode (asr_serve_*)");
  const asr_model_cfg& g = c->cfg;
  const int P = in->n_prefill, D = in->n_decode;
  if (P < 0 || P > g.max_prefill) return fail(ASR_EINVAL, "n_prefill out of [0, max_prefill]");
  if (D < 0 || D > g.max_decode) return fail(ASR_EINVAL, "n_decode out of [0, max_decode]");
  if (P > 0 && (!in->prefill_ids || !out->slot_of)) return fail(ASR_EINVAL, "NULL prefill arrays");
  if (D > 0 && (!in->slots || !in->tokens || !out->argmax || !out->done))
    return fail(ASR_EINVAL, "NULL decode arrays");
  if (P > 0 && g.n_enc == 0) return fail(ASR_EINVAL, "decoder-only context cannot prefill audio");
  if (D > 0 && g.n_dec == 0) return fail(ASR_EINVAL, "encoder-only context cannot decode");
  // validate prefill
  std::vector<int> taken;
  std::vector<const Request*> reqs;
  for (int i = 0; i < P; ++i) {
    auto it = c->popped.find(in->prefill_ids[i]);
    if (it == c->popped.end())
      return fail(ASR_EINVAL, "prefill id " + std::to_string(in->prefill_ids[i]) + " was not popped");
    if (!it->second.has_audio) return fail(ASR_EINVAL, "request without samples cannot be prefilled");
    for (int j = 0; j < i; ++j)
      if (in->prefill_ids[j] == in->prefill_ids[i]) return fail(ASR_EINVAL, "duplicate prefill id");
    int s = free_slot(c, taken);
    if (s < 0) return fail(ASR_EFULL, "no free decode slot");
    taken.push_back(s);
    reqs.push_back(&it->second);
  }
  // validate decode rows (slots being prefilled now count as occupied at position 0)
  std::vector<int32_t> pos(D);
  for (int i = 0; i < D; ++i) {
    int s = in->slots[i];
    if (s < 0 || s >= g.max_slots) return fail(ASR_EINVAL, "decode slot out of range");
    bool pre = std::find(taken.begin(), taken.end(), s) != taken.end();
    if (!pre && !c->slots[s].occupied) return fail(ASR_EINVAL, "decode slot not occupied");
    for (int j = 0; j < i; ++j)
      if (in->slots[j] == s) return fail(ASR_EINVAL, "duplicate decode slot");
    if (in->tokens[i] < 0 || in->tokens[i] >= g.vocab) return fail(ASR_EINVAL, "token id out of range");
    pos[i] = pre ? 0 : c->slots[s].pos;
    if (pos[i] >= kTextCtx) return fail(ASR_EINVAL, "slot position reached 448");
  }
  HIPCHK(hipSetDevice(c->device));
  if (P > 0) {
    std::vector<int32_t> sl(taken.begin(), taken.end());
    st = run_prefill(c, reqs, sl);
    if (st != ASR_OK) return st;
    for (int i = 0; i < P; ++i) {
      Slot& sl2 = c->slots[taken[i]];
      sl2.occupied = 1;
      sl2.id = reqs[i]->id;
      sl2.pos = 0;
      sl2.steps_left = steps_for(reqs[i]->n_samples, reqs[i]->max_tokens);
      out->slot_of[i] = taken[i];
      c->popped.erase(reqs[i]->id);
    }
  }
  if (D > 0) {
    asr_status dst = run_decode(c, D, in->slots, in->tokens, pos, out->argmax, in->logits);
    if (dst != ASR_OK && dst != ASR_EDEVICE) return dst;
    for (int i = 0; i < D; ++i) {
      Slot& sl2 = c->slots[in->slots[i]];
      sl2.pos += 1;
      if (sl2.steps_left > 0) sl2.steps_left -= 1;
      out->done[i] = sl2.steps_left == 0;
    }
    if (dst != ASR_OK) return dst;
  }
  return collect_timing(c);
}

// ---------------------------------------------------------------------------
// Continuous batching
// ---------------------------------------------------------------------------
asr_status asr_serve_config(asr_ctx* c, const asr_serve_cfg* sc) {
  if (!c || !sc) return fail(ASR_EINVAL, "NULL argument");
  if (!c->popped.empty()) return fail(ASR_ESTATE, "popped requests are waiting for asr_step");
  for (const auto& sl : c->slots)
    if (sl.occupied) return fail(ASR_ESTATE, "slots are occupied (release them first)");
  if (c->serve.busy()) return fail(ASR_ESTATE, "requests are still being served");
  const asr_model_cfg& g = c->cfg;
  const int n_slots = c->device >= 0 ? std::min(g.max_slots, g.max_decode) : g.max_slots;
  if (n_slots <= 0) return fail(ASR_EINVAL, "context has no decode slots");
  if (sc->max_admit < 1 || (c->device >= 0 && sc->max_admit > g.max_prefill))
    return fail(ASR_EINVAL, "max_admit out of [1, max_prefill]");
  if (sc->cross_tokens < 0) return fail(ASR_EINVAL, "cross_tokens must be >= 0");
  if (sc->tok_num <= 0 || sc->tok_den <= 0) return fail(ASR_EINVAL, "token rate must be positive");
  if (c->device >= 0 && (sc->start_token < 0 || sc->start_token >= g.vocab))
    return fail(ASR_EINVAL, "start_token out of the vocabulary");
  ServeConfig cfg;
  cfg.tok_num = sc->tok_num;
  cfg.tok_den = sc->tok_den;
  if (sc->kv_capacity > 0) {
    // every request must fit the pool on its own, or it could never finish
    ServeEngine probe;
    probe.configure(cfg);
    for (const auto& kv : c->waiting) {
      const Request& r = kv.second;
      QEntry e{r.id, r.arrival_us, r.n_samples, r.dur_us, r.sample_rate, r.max_tokens, 0};
      if ((int64_t)sc->cross_tokens + probe.tokens_for(e) > sc->kv_capacity)
        return fail(ASR_EINVAL, "request " + std::to_string(r.id) + " can never fit the KV pool");
    }
  }
  if (sc->dynamic && (sc->depth_low < 0 || sc->starve_num < 0 || sc->starve_den <= 0))
    return fail(ASR_EINVAL, "dynamic policy: depth_low >= 0, starve_num >= 0, starve_den > 0");
  c->serve_overlap = sc->overlap != 0;
  c->overlap_reserve = sc->overlap > 1 ? sc->overlap : 0;
  cfg.defer_first = sc->overlap != 0;
  cfg.dynamic = sc->dynamic != 0;
  cfg.depth_low = sc->depth_low;
  cfg.starve_num = sc->starve_num;
  cfg.starve_den = sc->dynamic ? sc->starve_den : 1;
  cfg.n_slots = n_slots;
  cfg.max_admit = sc->max_admit;
  cfg.kv_capacity = sc->kv_capacity;
  cfg.cross_tokens = sc->cross_tokens;
  cfg.tok_num = sc->tok_num;
  cfg.tok_den = sc->tok_den;
  cfg.start_token = sc->start_token;
  c->serve.configure(cfg);
  c->serving.clear();
  c->serve_mode = true;
  return ASR_OK;
}

}  // extern "C"

namespace {

// Plan one engine step and move the request records with it.
asr_status serve_plan_step(asr_ctx* c, int64_t now_us, const asr_serve_out* out, ServePlan* p) {
  if (!c->serve_mode) return fail(ASR_ESTATE, "asr_serve_config has not been called");
  if (!out || out->cap < c->serve.config().n_slots || !out->preempted || !out->admitted ||
      !out->admitted_slot || !out->decoded || !out->token || !out->finished)
    return fail(ASR_EINVAL, "asr_serve_out needs arrays of at least the slot count");
  *p = c->serve.plan(now_us, c->queue);
  for (int64_t id : p->preempted) {
    auto it = c->serving.find(id);
    c->waiting.emplace(id, std::move(it->second));
    c->serving.erase(it);
  }
  for (int64_t id : p->admitted) {
    auto it = c->waiting.find(id);
    c->serving.emplace(id, std::move(it->second));
    c->waiting.erase(it);
  }
  return ASR_OK;
}

void serve_finish(asr_ctx* c, const ServePlan& p, const int32_t* tokens, asr_serve_out* out) {
  std::vector<int64_t> fin = c->serve.commit(p, tokens);
  out->policy = p.policy;
  out->n_preempted = (int32_t)p.preempted.size();
  for (size_t i = 0; i < p.preempted.size(); ++i) out->preempted[i] = p.preempted[i];
  out->n_admitted = (int32_t)p.admitted.size();
  for (size_t i = 0; i < p.admitted.size(); ++i) {
    out->admitted[i] = p.admitted[i];
    out->admitted_slot[i] = p.admitted_slot[i];
  }
  out->n_decoded = (int32_t)p.dec_id.size();
  for (size_t i = 0; i < p.dec_id.size(); ++i) {
    out->decoded[i] = p.dec_id[i];
    out->token[i] = tokens ? tokens[i] : -1;
  }
  out->n_finished = (int32_t)fin.size();
  for (size_t i = 0; i < fin.size(); ++i) {
    out->finished[i] = fin[i];
    c->serving.erase(fin[i]);
  }
  // mirror the engine into the slot table (asr_slot_info)
  for (auto& sl : c->slots) sl = Slot();
  for (size_t i = 0; i < p.dec_id.size(); ++i) {
    const RunEntry* r = c->serve.find(p.dec_id[i]);
    if (!r) continue;
    Slot& sl = c->slots[r->slot];
    sl.occupied = 1;
    sl.id = r->q.id;
    sl.pos = r->generated;
    sl.steps_left = r->total - r->generated;
  }
}

}  // namespace

extern "C" {

asr_status asr_serve_plan(asr_ctx* c, int64_t now_us, asr_serve_out* out) {
  if (!c) return fail(ASR_EINVAL, "NULL context");
  if (c->device >= 0)
    return fail(ASR_ESTATE, "asr_serve_plan runs the schedule without the model: queue-only contexts");
  ServePlan p;
  asr_status st = serve_plan_step(c, now_us, out, &p);
  if (st != ASR_OK) return st;
  serve_finish(c, p, nullptr, out);
  return ASR_OK;
}

asr_status asr_serve_step(asr_ctx* c, int64_t now_us, asr_serve_out* out) {
  asr_status st = need_gpu(c, true);
  if (st != ASR_OK) return st;
  if (c->cfg.n_enc == 0 || c->cfg.n_dec == 0)
    return fail(ASR_EINVAL, "continuous batching needs an encoder and a decoder");
  ServePlan p;
  st = serve_plan_step(c, now_us, out, &p);
  if (st != ASR_OK) return st;
  HIPCHK(hipSetDevice(c->device));
  std::vector<const Request*> reqs;
  for (int64_t id : p.admitted) {
    const Request& r = c->serving.at(id);
    if (!r.has_audio) return fail(ASR_EINVAL, "request " + std::to_string(id) + " has no samples");
    reqs.push_back(&r);
  }
  const int D = (int)p.dec_id.size(), A = (int)p.admitted.size();
  std::vector<int32_t> tok(D);
  if (c->serve_overlap && A > 0 && D > 0) {
    // With overlap the engine defers an admitted request's first token to
    // the next step, so this step's decode rows do not depend on its prefill:
    // the prefill runs on a second stream while the rows decode on the bound
    // stream.  The two share only read-only weights and disjoint slots.
    if (!c->pstream) {
      HIPCHK(hipStreamCreateWithFlags(&c->pstream, hipStreamNonBlocking));
      HIPCHK(hipEventCreateWithFlags(&c->ev_fork, hipEventDisableTiming));
      HIPCHK(hipEventCreateWithFlags(&c->ev_join, hipEventDisableTiming));
    }
    hipStream_t main_stream = c->stream;
    HIPCHK(hipEventRecord(c->ev_fork, main_stream));
    HIPCHK(hipStreamWaitEvent(c->pstream, c->ev_fork, 0));
    PrefillStage stage;
    c->stream = c->pstream;
    gemm_set_cu_reserve(c->overlap_reserve);
    st = launch_prefill(c, reqs, p.admitted_slot, stage);
    gemm_set_cu_reserve(0);
    c->stream = main_stream;
    if (st == ASR_OK)
      st = run_decode(c, D, p.dec_slot.data(), p.dec_token.data(), p.dec_pos, tok.data(), nullptr);
    HIPCHK(hipStreamSynchronize(c->pstream));    // the prefill and its stage's host arrays
    if (st != ASR_OK) return st;
  } else {
    st = run_prefill(c, reqs, p.admitted_slot);
    if (st != ASR_OK) return st;
    st = run_decode(c, D, p.dec_slot.data(), p.dec_token.data(), p.dec_pos, tok.data(), nullptr);
    if (st != ASR_OK) return st;
  }
  serve_finish(c, p, tok.data(), out);
  return collect_timing(c);
}

asr_status asr_serve_simulate(asr_ctx* c, const asr_sim_cost* cost, int64_t t0_us, int32_t n,
                              const int64_t* ids, int64_t* first_us, int64_t* finish_us,
                              int32_t* n_tokens, int32_t* n_preempt, int64_t* token_us,
                              int64_t token_cap, int64_t* t_end_us) {
  if (!c || !cost || (n > 0 && (!ids || !first_us || !finish_us || !n_tokens || !n_preempt)) ||
      !t_end_us)
    return fail(ASR_EINVAL, "NULL argument");
  if (c->device >= 0) return fail(ASR_ESTATE, "simulations run on queue-only contexts");
  if (!c->serve_mode) return fail(ASR_ESTATE, "asr_serve_config has not been called");
  if (cost->prefill_us < 0 || cost->step_us < 0 || cost->row_us < 0 ||
      cost->prefill_us + cost->step_us + cost->row_us <= 0)
    return fail(ASR_EINVAL, "step costs must be >= 0 and not all zero");
  if (c->serve.busy()) return fail(ASR_ESTATE, "requests are already being served");
  if ((size_t)n != c->waiting.size()) return fail(ASR_EINVAL, "ids must list every submitted request");
  std::unordered_map<int64_t, int32_t> idx;
  int64_t off = 0;
  std::vector<int64_t> tok_off(n);
  for (int32_t i = 0; i < n; ++i) {
    auto it = c->waiting.find(ids[i]);
    if (it == c->waiting.end() || idx.count(ids[i]))
      return fail(ASR_EINVAL, "id " + std::to_string(ids[i]) + " is not a distinct waiting request");
    idx[ids[i]] = i;
    const Request& r = it->second;
    QEntry e{r.id, r.arrival_us, r.n_samples, r.dur_us, r.sample_rate, r.max_tokens, 0};
    tok_off[i] = off;
    off += c->serve.tokens_for(e);
    first_us[i] = finish_us[i] = -1;
    n_tokens[i] = n_preempt[i] = 0;
  }
  if (token_us && token_cap < off) return fail(ASR_EINVAL, "token_us needs room for every token");
  int64_t t = t0_us;
  int32_t left = n;
  asr_serve_out dummy{};
  std::vector<int32_t> gen;
  while (left > 0) {
    if (!c->serve.busy() && !c->queue.any_eligible(t)) {
      t = c->queue.min_arrival();
      continue;
    }
    ServePlan p = c->serve.plan(t, c->queue);
    for (int64_t id : p.preempted) {
      auto it = c->serving.find(id);
      c->waiting.emplace(id, std::move(it->second));
      c->serving.erase(it);
      n_preempt[idx[id]] += 1;
    }
    for (int64_t id : p.admitted) {
      auto it = c->waiting.find(id);
      c->serving.emplace(id, std::move(it->second));
      c->waiting.erase(it);
    }
    const int64_t nd = (int64_t)p.dec_id.size();
    t += cost->prefill_us * (int64_t)p.admitted.size() +
         (nd > 0 ? cost->step_us + cost->row_us * nd : 0);
    std::vector<int64_t> fin = c->serve.commit(p, nullptr, &gen);
    for (size_t i = 0; i < p.dec_id.size(); ++i) {
      const int32_t k = idx[p.dec_id[i]];
      // a position that a recomputed request reaches again is not emitted again
      while (n_tokens[k] < gen[i]) {
        if (token_us) token_us[tok_off[k] + n_tokens[k]] = t;
        if (n_tokens[k] == 0) first_us[k] = t;
        n_tokens[k] += 1;
      }
    }
    for (int64_t id : fin) {
      finish_us[idx[id]] = t;
      c->serving.erase(id);
      (void)c->serve.take_result(id, nullptr);
      --left;
    }
    (void)dummy;
  }
  *t_end_us = t;
  return ASR_OK;
}

asr_status asr_serve_stats(const asr_ctx* c, int64_t steps[3]) {
  if (!c || !steps) return fail(ASR_EINVAL, "NULL argument");
  for (int k = 0; k < 3; ++k) steps[k] = c->serve.steps_under(k);
  return ASR_OK;
}

asr_status asr_serve_tokens(asr_ctx* c, int64_t id, int32_t* tokens, int32_t cap, int32_t* n) {
  if (!c || !n || (cap > 0 && !tokens)) return fail(ASR_EINVAL, "NULL argument");
  std::vector<int32_t> t;
  if (!c->serve.take_result(id, &t)) return fail(ASR_ENOTFOUND, "no finished request " + std::to_string(id));
  if ((int32_t)t.size() > cap) return fail(ASR_EINVAL, "token buffer too small");
  for (size_t i = 0; i < t.size(); ++i) tokens[i] = t[i];
  *n = (int32_t)t.size();
  return ASR_OK;
}

asr_status asr_set_decode_graphs(asr_ctx* c, int32_t on) {
  if (!c) return fail(ASR_EINVAL, "NULL context");
  c->decode_graphs = on != 0;
  return ASR_OK;
}

asr_status asr_set_encoder_streams(asr_ctx* c, int32_t n) {
  if (!c) return fail(ASR_EINVAL, "NULL context");
  if (n < 1 || n > asr_ctx::kEncGroups) return fail(ASR_EINVAL, "n out of [1, 4]");
  c->enc_groups = n;
  return ASR_OK;
}

asr_status asr_set_timing(asr_ctx* c, int32_t classes) {
  if (!c) return fail(ASR_EINVAL, "NULL context");
  if (c->device < 0) return fail(ASR_ENODEV, "queue-only context");
  if (classes & ~ASR_TIME_ALL) return fail(ASR_EINVAL, "unknown timing class bits");
  c->timing = classes;
  return ASR_OK;
}

asr_status asr_reset_timing(asr_ctx* c) {
  if (!c) return fail(ASR_EINVAL, "NULL context");
  asr_status st = c->device >= 0 ? collect_timing(c) : ASR_OK;
  for (int i = 0; i < ASR_K_COUNT; ++i) c->t_ms[i] = c->t_flops[i] = c->t_bytes[i] = 0, c->t_n[i] = 0;
  return st;
}

asr_status asr_get_timing(asr_ctx* c, int32_t cls, double* ms, int64_t* launches, double* flops,
                          double* bytes) {
  if (!c) return fail(ASR_EINVAL, "NULL context");
  if (cls < 0 || cls >= ASR_K_COUNT) return fail(ASR_EINVAL, "kernel class");
  if (c->device >= 0) {
    asr_status st = collect_timing(c);
    if (st != ASR_OK) return st;
  }
  if (ms) *ms = c->t_ms[cls];
  if (launches) *launches = c->t_n[cls];
  if (flops) *flops = c->t_flops[cls];
  if (bytes) *bytes = c->t_bytes[cls];
  return ASR_OK;
}

asr_status asr_debug_logmel(asr_ctx* c, const float* const* pcm, const int64_t* n_samples, int32_t n,
                            int32_t on_device, float* out) {
  asr_status st = need_gpu(c, false);
  if (st != ASR_OK) return st;
  if (!pcm || !n_samples || !out) return fail(ASR_EINVAL, "NULL argument");
  if (n <= 0 || n > c->cfg.max_prefill) return fail(ASR_EINVAL, "n out of [1, max_prefill]");
  HIPCHK(hipSetDevice(c->device));
  st = stage_pcm(c, pcm, n_samples, n, on_device != 0);
  if (st != ASR_OK) return st;
  st = run_mel(c, n);
  if (st != ASR_OK) return st;
  float* tmp = c->at<float>(c->L.wstage);
  mel_normalize<float>(c->at<float>(c->L.mel_raw), c->at<float>(c->L.mel_gmax), n,
                       c->cfg.n_mels, tmp, 0, c->stream);
  CHECK_LAUNCH();
  HIPCHK(hipMemcpyAsync(out, tmp, (size_t)n * kFrames * c->cfg.n_mels * 4, hipMemcpyDeviceToHost,
                        c->stream));
  HIPCHK(hipStreamSynchronize(c->stream));
  return collect_timing(c);
}

asr_status asr_debug_encode(asr_ctx* c, const float* const* pcm, const int64_t* n_samples, int32_t n,
                            int32_t on_device, float* out) {
  asr_status st = need_gpu(c, true);
  if (st != ASR_OK) return st;
  if (!pcm || !n_samples || !out) return fail(ASR_EINVAL, "NULL argument");
  if (n <= 0 || n > c->cfg.max_prefill) return fail(ASR_EINVAL, "n out of [1, max_prefill]");
  if (c->cfg.n_enc == 0) return fail(ASR_EINVAL, "decoder-only context");
  HIPCHK(hipSetDevice(c->device));
  st = stage_pcm(c, pcm, n_samples, n, on_device != 0);
  if (st != ASR_OK) return st;
  st = c->bf16() ? encode_clips<bf16_t>(c, n) : encode_clips<float>(c, n);
  if (st != ASR_OK) return st;
  const int64_t cnt = (int64_t)n * kCtx * c->cfg.d_model;
  float* tmp = c->at<float>(c->L.wstage);
  if (c->bf16())
    convert_to_f32<bf16_t>(c->at<bf16_t>(c->L.xn), tmp, cnt, c->stream);
  else
    convert_to_f32<float>(c->at<float>(c->L.xn), tmp, cnt, c->stream);
  CHECK_LAUNCH();
  HIPCHK(hipMemcpyAsync(out, tmp, cnt * 4, hipMemcpyDeviceToHost, c->stream));
  HIPCHK(hipStreamSynchronize(c->stream));
  return collect_timing(c);
}

asr_status asr_debug_attention(asr_ctx* c, const float* q, const float* k, const float* v,
                               int32_t n, float* out) {
  asr_status st = need_gpu(c, true);
  if (st != ASR_OK) return st;
  if (!q || !k || !v || !out) return fail(ASR_EINVAL, "NULL argument");
  if (n <= 0 || n > c->cfg.max_prefill) return fail(ASR_EINVAL, "n out of [1, max_prefill]");
  if (c->cfg.n_enc == 0) return fail(ASR_EINVAL, "decoder-only context");
  HIPCHK(hipSetDevice(c->device));
  const Layout& L = c->L;
  const int d = c->cfg.d_model, H = c->cfg.n_head, R = n * kCtx;
  const int64_t cnt = (int64_t)R * d;
  float* tmp = c->at<float>(L.wstage);
  const float* src[3] = {q, k, v};
  for (int which = 0; which < 3; ++which) {
    HIPCHK(hipMemcpyAsync(tmp, src[which], cnt * 4, hipMemcpyHostToDevice, c->stream));
    // the bf16 kernel takes q in the exp2 domain as given; the fp32 kernel
    // applies 1/sqrt(64) itself and uses exp, so it gets q * 8 / log2(e)
    if (c->bf16())
      pack_attn_operand<bf16_t>(tmp, which, R, d, H, 1.0f, c->at<bf16_t>(L.qkv),
                                c->at<bf16_t>(L.vt), c->stream);
    else
      pack_attn_operand<float>(tmp, which, R, d, H, 1.0f / kQScaleLog2, c->at<float>(L.qkv),
                               nullptr, c->stream);
  }
  if (c->bf16()) {
    flash_attn_bf16(c->at<bf16_t>(L.qkv), c->at<bf16_t>(L.vt), c->at<bf16_t>(L.att), n, H,
                    c->stream);
    convert_to_f32<bf16_t>(c->at<bf16_t>(L.att), tmp, cnt, c->stream);
  } else {
    flash_attn_f32(c->at<float>(L.qkv), c->at<float>(L.att), n, H, c->stream);
    convert_to_f32<float>(c->at<float>(L.att), tmp, cnt, c->stream);
  }
  CHECK_LAUNCH();
  HIPCHK(hipMemcpyAsync(out, tmp, cnt * 4, hipMemcpyDeviceToHost, c->stream));
  HIPCHK(hipStreamSynchronize(c->stream));
  return ASR_OK;
}

asr_status asr_debug_set_encoder_out(asr_ctx* c, const int32_t* slots, const int64_t* ids,
                                     const int32_t* steps_left, int32_t n, const float* E,
                                     int32_t on_device) {
  asr_status st = need_gpu(c, true);
  if (st != ASR_OK) return st;
  if (!slots || !ids || !steps_left || !E) return fail(ASR_EINVAL, "NULL argument");
  if (n <= 0 || n > std::max(1, c->cfg.max_prefill)) return fail(ASR_EINVAL, "n out of [1, max_prefill]");
  if (c->cfg.n_dec == 0) return fail(ASR_EINVAL, "encoder-only context");
  for (int i = 0; i < n; ++i) {
    if (slots[i] < 0 || slots[i] >= c->cfg.max_slots) return fail(ASR_EINVAL, "slot out of range");
    for (int j = 0; j < i; ++j)
      if (slots[j] == slots[i]) return fail(ASR_EINVAL, "duplicate slot");
    if (ids[i] >= 0 && !c->popped.count(ids[i])) return fail(ASR_EINVAL, "id was not popped");
    if (steps_left[i] < 1 || steps_left[i] > kTextCtx) return fail(ASR_EINVAL, "steps_left out of [1, 448]");
  }
  HIPCHK(hipSetDevice(c->device));
  hipStream_t s = c->stream;
  const int d = c->cfg.d_model;
  const int64_t cnt = (int64_t)n * kCtx * d;
  // E goes through the f32 staging area into the storage-typed activation buffer
  float* tmp = c->at<float>(c->L.wstage);
  if ((int64_t)c->L.wstage_floats < cnt) return fail(ASR_EINVAL, "too many clips for staging");
  HIPCHK(hipMemcpyAsync(tmp, E, cnt * 4, on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice, s));
  if (c->bf16())
    convert_from_f32<bf16_t>(tmp, c->at<bf16_t>(c->L.xn), cnt, s);
  else
    convert_from_f32<float>(tmp, c->at<float>(c->L.xn), cnt, s);
  HIPCHK(hipMemcpyAsync(c->at(c->L.p_slots), slots, n * 4, hipMemcpyHostToDevice, s));
  st = c->bf16() ? cross_kv<bf16_t>(c, c->at(c->L.xn), n, 0) : cross_kv<float>(c, c->at(c->L.xn), n, 0);
  if (st != ASR_OK) return st;
  HIPCHK(hipStreamSynchronize(s));
  for (int i = 0; i < n; ++i) {
    Slot& sl = c->slots[slots[i]];
    sl.occupied = 1;
    sl.id = ids[i];
    sl.pos = 0;
    sl.steps_left = steps_left[i];
    if (ids[i] >= 0) c->popped.erase(ids[i]);
  }
  return collect_timing(c);
}

asr_status asr_debug_get_kv(asr_ctx* c, int32_t slot, int32_t which, float* out) {
  asr_status st = need_gpu(c, false);
  if (st != ASR_OK) return st;
  if (!out) return fail(ASR_EINVAL, "NULL argument");
  if (slot < 0 || slot >= c->cfg.max_slots) return fail(ASR_EINVAL, "slot out of range");
  if (which != 0 && which != 1) return fail(ASR_EINVAL, "which must be 0 (self) or 1 (cross)");
  HIPCHK(hipSetDevice(c->device));
  const int64_t cnt = which == 0 ? c->L.self_stride : c->L.cross_stride;
  const size_t off = (which == 0 ? c->L.self_kv : c->L.cross_kv) + (size_t)slot * cnt * c->es;
  float* tmp = c->at<float>(c->L.wstage);
  if (c->bf16())
    convert_to_f32<bf16_t>(c->at<bf16_t>(off), tmp, cnt, c->stream);
  else
    convert_to_f32<float>(c->at<float>(off), tmp, cnt, c->stream);
  CHECK_LAUNCH();
  HIPCHK(hipMemcpyAsync(out, tmp, cnt * 4, hipMemcpyDeviceToHost, c->stream));
  HIPCHK(hipStreamSynchronize(c->stream));
  return ASR_OK;
}

asr_status asr_debug_set_self_kv(asr_ctx* c, int32_t slot, const float* src, int32_t length,
                                 int32_t on_device) {
  asr_status st = need_gpu(c, false);
  if (st != ASR_OK) return st;
  if (!src) return fail(ASR_EINVAL, "NULL argument");
  if (slot < 0 || slot >= c->cfg.max_slots) return fail(ASR_EINVAL, "slot out of range");
  if (!c->slots[slot].occupied) return fail(ASR_EINVAL, "slot not occupied");
  if (length < 0 || length >= kTextCtx) return fail(ASR_EINVAL, "length out of [0, 447]");
  HIPCHK(hipSetDevice(c->device));
  const int64_t cnt = c->L.self_stride;
  const size_t off = c->L.self_kv + (size_t)slot * cnt * c->es;
  float* tmp = c->at<float>(c->L.wstage);
  HIPCHK(hipMemcpyAsync(tmp, src, cnt * 4, on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice,
                        c->stream));
  if (c->bf16())
    convert_from_f32<bf16_t>(tmp, c->at<bf16_t>(off), cnt, c->stream);
  else
    convert_from_f32<float>(tmp, c->at<float>(off), cnt, c->stream);
  CHECK_LAUNCH();
  HIPCHK(hipStreamSynchronize(c->stream));
  c->slots[slot].pos = length;
  return ASR_OK;
}

}  // extern "C"

// ===========================================================================
// Allocation-free log-mel front-end (asr_logmel_noalloc)
//
// The scratch the front-end needs -- the window and twiddle tables, the mel
// filterbanks of both supported widths with their bin ranges, and the
// per-clip maxima of one call -- lives in a file-scope device array instead
// of a bound block.  Host code never names that array directly: each device
// resolves its own copy's address once (hipGetSymbolAddress, with that
// device current) and every launch takes that address.
// ===========================================================================
namespace {

constexpr int kNaDevices = 64;
// word offsets into the scratch array
constexpr size_t kNaWin = 0, kNaCos = kNaWin + kNFFT, kNaSin = kNaCos + kNFFT;
// (packed filter weights: every bin lies in at most two filters)
constexpr size_t kNaFb80 = kNaSin + kNFFT, kNaFb128 = kNaFb80 + 2 * kBins;
constexpr size_t kNaRng80 = kNaFb128 + 2 * kBins, kNaRng128 = kNaRng80 + 3 * 80;
constexpr size_t kNaMax = kNaRng128 + 3 * 128;   // group maxima [clips][kMelGroups]
constexpr size_t kNaWords = kNaMax + (size_t)kMelArgClips * kMelGroups;
constexpr size_t kNaBytes = 64 * 1024;   // the stated maximum: 64 KiB per GPU
static_assert(kNaWords * 4 <= kNaBytes, "scratch layout");

}  // namespace

static __device__ __align__(256) uint32_t scratch[kNaBytes / 4];

namespace {

std::mutex g_na_mu;
uint32_t* g_na_ptr[kNaDevices] = {};

// First call on a device (that device current): resolve the array's address
// and upload the constant tables with synchronous copies.
asr_status na_setup(int dev, uint32_t** out) {
  std::lock_guard<std::mutex> lock(g_na_mu);
  if (!g_na_ptr[dev]) {
    void* p = nullptr;
    HIPCHK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(ASR_EDEVICE, "hipGetSymbolAddress returned NULL");
    uint32_t* base = (uint32_t*)p;
    const HostMelTables t80 = host_mel_tables(80), t128 = host_mel_tables(128);
    if (t80.fb.size() > 2 * kBins || t128.fb.size() > 2 * kBins)
      return fail(ASR_EINVAL, "packed filterbank larger than two weights per bin");
    HIPCHK(hipMemcpy(base + kNaWin, t80.win.data(), kNFFT * 4, hipMemcpyHostToDevice));
    HIPCHK(hipMemcpy(base + kNaCos, t80.ct.data(), kNFFT * 4, hipMemcpyHostToDevice));
    HIPCHK(hipMemcpy(base + kNaSin, t80.st.data(), kNFFT * 4, hipMemcpyHostToDevice));
    HIPCHK(hipMemcpy(base + kNaFb80, t80.fb.data(), t80.fb.size() * 4, hipMemcpyHostToDevice));
    HIPCHK(hipMemcpy(base + kNaFb128, t128.fb.data(), t128.fb.size() * 4, hipMemcpyHostToDevice));
    HIPCHK(hipMemcpy(base + kNaRng80, t80.rng.data(), t80.rng.size() * 4, hipMemcpyHostToDevice));
    HIPCHK(hipMemcpy(base + kNaRng128, t128.rng.data(), t128.rng.size() * 4,
                     hipMemcpyHostToDevice));
    g_na_ptr[dev] = base;
  }
  *out = g_na_ptr[dev];
  return ASR_OK;
}

}  // namespace

extern "C" asr_status asr_logmel_noalloc(const float* const* pcm, const int64_t* n_samples,
                                         int32_t n, int32_t n_mels, float* out, void* stream) {
  if (!pcm || !n_samples || !out) return fail(ASR_EINVAL, "NULL argument");
  if (n < 1 || n > kMelArgClips)
    return fail(ASR_EINVAL, "n out of [1, " + std::to_string(kMelArgClips) + "] (scratch limit)");
  if (n_mels != 80 && n_mels != 128) return fail(ASR_EINVAL, "n_mels must be 80 or 128");
  MelClipArgs clips{};
  for (int i = 0; i < n; ++i) {
    if (n_samples[i] < 0 || n_samples[i] > kSamples30s)
      return fail(ASR_EINVAL, "n_samples out of [0, 480000]");
    if (n_samples[i] > 0 && !pcm[i]) return fail(ASR_EINVAL, "NULL pcm");
    clips.ptr[i] = pcm[i];
    clips.n[i] = n_samples[i];
  }
  int dev = -1;
  HIPCHK(hipGetDevice(&dev));
  if (dev < 0 || dev >= kNaDevices) return fail(ASR_EINVAL, "device index out of range");
  uint32_t* base = nullptr;
  asr_status st = na_setup(dev, &base);
  if (st != ASR_OK) return st;
  const bool wide = n_mels == 128;
  MelTables t{(const float*)(base + kNaWin), (const float*)(base + kNaCos),
              (const float*)(base + kNaSin), (const float*)(base + (wide ? kNaFb128 : kNaFb80)),
              (const int32_t*)(base + (wide ? kNaRng128 : kNaRng80))};
  hipStream_t s = (hipStream_t)stream;
  // raw log-mel straight into out, then the clamp and affine in place
  float* gmax = (float*)(base + kNaMax);
  log_mel_args(clips, n, n_mels, t, out, gmax, s);
  mel_normalize<float>(out, gmax, n, n_mels, out, 0, s);
  CHECK_LAUNCH();
  return ASR_OK;
}
