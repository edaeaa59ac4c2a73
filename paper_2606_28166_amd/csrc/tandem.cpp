// libtandem: C ABI and host runtime of the tandem co-generation step.
//
// One handle holds a senior and a junior decoder (borrowed device weights),
// one KV cache per model inside the caller's KV arena, activation and
// per-sequence state buffers inside the caller's scratch buffer, and the
// caller's stream.  A step forwards the pending token of every sequence
// through BOTH models (each appends to its own cache: the caches stay in
// lockstep with the shared history), samples the owner's next token,
// records (token, authorship bit, senior log-prob) and applies the handoff
// rule — the rollout half of Algorithm 1, one token at a time for all
// sequences of the batch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "tandem.h"
#include "kernels.h"

using namespace tandem;

namespace {

thread_local std::string g_err = "no error";

constexpr int kSplitMax = 16;         // split-K slices of a decode projection
constexpr int kVocabChunk = 4096;     // vocabulary entries per sampling workgroup
constexpr int kSampleParts = 1024;    // partials per row of the LM heads' sampling epilogue (>= their grid)
constexpr int kCompactEvery = 32;     // decode steps between compactions of the batch (EOS runs)
constexpr int kCompactBucket = 32;    // the launched row count is a multiple of this
constexpr size_t kAlign = 256;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct Layer {
  const float* attn_norm;
  const void* w_qkv;
  const float* q_norm;
  const float* k_norm;
  const void* w_o;
  const float* ffn_norm;
  const void* w_gate_up;
  const void* w_down;
  // packed copies (NULL: the matrix has none)
  const void* p_qkv;
  const void* p_o;
  const void* p_gate_up;
  const void* p_down;
};

struct ModelPlan {            // byte offsets / sizes of one model's buffers
  size_t esz;
  int qkv_dim, att_dim, rmax;
  size_t ws_floats;
  size_t kv_half;             // bytes of the K (= V) cache
  size_t off_h, off_xa, off_xf, off_q, off_ws, off_logits, off_rope;
  size_t off_packed, packed_bytes;   // MFMA-ordered copies of the projection and LM-head weights
};

// The matrices of a model in packing order: per layer QKV, O, gate/up, down,
// then the LM head.  (rows N, reduction length K)
std::vector<std::pair<int, int>> packed_shapes(const tandem_model_cfg* c) {
  std::vector<std::pair<int, int>> v;
  const int d = c->d_model, qkv = (c->n_q_heads + 2 * c->n_kv_heads) * c->head_dim, att = c->n_q_heads * c->head_dim;
  for (int l = 0; l < c->n_layers; ++l) {
    v.push_back({qkv, d});
    v.push_back({d, att});
    v.push_back({2 * c->ffn_dim, d});
    v.push_back({d, c->ffn_dim});
  }
  v.push_back({c->vocab, d});
  return v;
}

// A matrix gets a packed copy (and the streaming decode GEMM) when the model
// is bf16 and its shape fits that kernel.
bool packs(const tandem_model_cfg* c, int N, int K) {
  return c->weight_dtype == TANDEM_BF16 && c->ffn_dim % 16 == 0 && stream_gemm_ok(1, N, K);
}

struct Plan {
  int nm;                     // models: 2 (senior and junior), 1 (the senior alone)
  int ctx_stride;
  int n_chunks;
  ModelPlan m[2];
  size_t kv_bytes;
  size_t off_state, off_seq_slot, off_rows, off_prompt, off_partials, off_count, off_act, off_drows;
  size_t off_pfx;             // shared-prefix tables of the decode rows (2 x max_seqs int32)
  size_t off_err;             // the batch's token-range error flag (int32)
  size_t off_score;           // dual-distribution score partials [max_seqs][n_chunks][6]
  // Sampling inside the LM heads (both models' LM heads run as fp16 streaming
  // GEMMs): the step's Gumbel noise [noise_rows][vocab] and each head's
  // per-workgroup partials [noise_rows][kSampleParts][5]
  bool fused;
  int noise_rows;
  size_t off_noise, off_part_sen, off_part_jun;
  size_t scratch_bytes;
};

struct Model {
  tandem_model_cfg cfg;
  ModelPlan p;
  const void* embed;
  std::vector<Layer> layers;
  const float* final_norm;
  const void* lm_head;
  const void* p_lm;           // packed LM head (NULL: none)
  char* kc;
  char* vc;
  long layer_stride;          // elements
  long slot_stride;           // elements
  float* h;
  void* xa;                   // activation rows (split format for bf16 models; fp16 rows for the
  void* xf;                   // streaming FFN and LM-head products, see ffn16 / lm16)
  // The FFN projections (gate/up and down) and the LM head take fp16
  // activations and fp16 packed weights when they run on the streaming
  // decode GEMM; QKV and O keep the split format, whose precision the
  // attention (and the bf16-rounded K/V cache behind it) needs.
  bool ffn16 = false, lm16 = false;
  float* q;
  float* ws;
  float* logits;
  float2* rope;
};

tandem_status fail(std::string* where, tandem_status s, const std::string& msg) {
  if (where) *where = msg;
  g_err = msg;
  return s;
}

tandem_status check_cfg(const tandem_model_cfg* c, const char* who, std::string* err) {
  char b[256];
  if (c->n_layers < 1 || c->d_model < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1 || c->head_dim < 1 ||
      c->ffn_dim < 1 || c->vocab < 2) {
    snprintf(b, sizeof b, "%s: every size must be positive (vocab >= 2)", who);
    return fail(err, TANDEM_E_SHAPE, b);
  }
  if (c->n_q_heads % c->n_kv_heads != 0) {
    snprintf(b, sizeof b, "%s: n_q_heads (%d) must be a multiple of n_kv_heads (%d)", who, c->n_q_heads,
             c->n_kv_heads);
    return fail(err, TANDEM_E_SHAPE, b);
  }
  if (c->weight_dtype != TANDEM_BF16 && c->weight_dtype != TANDEM_F32) {
    snprintf(b, sizeof b, "%s: weight_dtype must be TANDEM_BF16 or TANDEM_F32", who);
    return fail(err, TANDEM_E_ARG, b);
  }
  if (c->head_dim != 32 && c->head_dim != 64 && c->head_dim != 128) {
    snprintf(b, sizeof b, "%s: head_dim %d unsupported (32, 64 or 128)", who, c->head_dim);
    return fail(err, TANDEM_E_UNSUPPORTED, b);
  }
  if (c->d_model % 8 || c->ffn_dim % 8) {
    snprintf(b, sizeof b, "%s: d_model and ffn_dim must be multiples of 8", who);
    return fail(err, TANDEM_E_UNSUPPORTED, b);
  }
  if (c->d_model > 8192 || (long)(c->n_q_heads + 2 * c->n_kv_heads) * c->head_dim > 16384) {
    snprintf(b, sizeof b, "%s: d_model <= 8192 and (n_q + 2 n_kv) * head_dim <= 16384 required", who);
    return fail(err, TANDEM_E_UNSUPPORTED, b);
  }
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f) || !std::isfinite(c->rope_theta)) {
    snprintf(b, sizeof b, "%s: rms_eps must be >= 0 and rope_theta finite and > 0", who);
    return fail(err, TANDEM_E_ARG, b);
  }
  return TANDEM_OK;
}

tandem_status check_cap(const tandem_capacity* cap, std::string* err) {
  if (cap->max_seqs < 1 || cap->max_ctx < 1 || cap->max_prefill_tokens < 1)
    return fail(err, TANDEM_E_CAPACITY, "capacity: max_seqs, max_ctx and max_prefill_tokens must be >= 1");
  if (cap->max_ctx > (1 << 24) || cap->max_seqs > (1 << 24) || cap->max_prefill_tokens > (1 << 24))
    return fail(err, TANDEM_E_CAPACITY, "capacity: sizes above 2^24 are not supported");
  return TANDEM_OK;
}

// Narrow FFNs give the fused gate/up + SwiGLU GEMM too few output tiles to
// fill the device: those run as a split-K GEMM over the 2 ffn gate and up
// rows plus a SwiGLU pass over the summed partials.
bool split_gate_up(const tandem_model_cfg* c) {
  return c->weight_dtype == TANDEM_BF16 && c->d_model % 64 == 0 && c->ffn_dim < 8192;
}

Plan make_plan(const tandem_model_cfg* sen, const tandem_model_cfg* jun, const tandem_capacity* cap) {
  Plan P{};
  P.ctx_stride = (int)align_up((size_t)cap->max_ctx, 64);
  P.n_chunks = (sen->vocab + kVocabChunk - 1) / kVocabChunk;
  const tandem_model_cfg* cf[2] = {sen, jun};
  P.nm = jun ? 2 : 1;
  size_t kv = 0, sc = 0;
  for (int i = 0; i < P.nm; ++i) {
    const tandem_model_cfg* c = cf[i];
    ModelPlan& m = P.m[i];
    m.esz = c->weight_dtype == TANDEM_BF16 ? 2 : 4;
    m.qkv_dim = (c->n_q_heads + 2 * c->n_kv_heads) * c->head_dim;
    m.att_dim = c->n_q_heads * c->head_dim;
    m.rmax = cap->max_seqs > cap->max_prefill_tokens ? cap->max_seqs : cap->max_prefill_tokens;
    size_t nmax = (size_t)(m.qkv_dim > c->d_model ? m.qkv_dim : c->d_model);
    if ((split_gate_up(c) || c->weight_dtype == TANDEM_BF16) && (size_t)2 * c->ffn_dim > nmax)
      nmax = (size_t)2 * c->ffn_dim;
    const size_t rows_ws = (size_t)kSplitMax * cap->max_seqs > (size_t)cap->max_prefill_tokens
                               ? (size_t)kSplitMax * cap->max_seqs
                               : (size_t)cap->max_prefill_tokens;
    m.ws_floats = rows_ws * nmax;
    m.kv_half = align_up((size_t)c->n_layers * cap->max_seqs * c->n_kv_heads * P.ctx_stride * c->head_dim * m.esz,
                         kAlign);
    kv += 2 * m.kv_half;
    const size_t R = (size_t)m.rmax;
    const size_t xa_w = (size_t)(m.att_dim > c->d_model ? m.att_dim : c->d_model);
    m.off_h = sc; sc = align_up(sc + R * c->d_model * 4, kAlign);
    m.off_xa = sc; sc = align_up(sc + R * xa_w * 4, kAlign);
    m.off_xf = sc; sc = align_up(sc + R * c->ffn_dim * 4, kAlign);
    m.off_q = sc; sc = align_up(sc + R * m.att_dim * 4, kAlign);
    m.off_ws = sc; sc = align_up(sc + m.ws_floats * 4, kAlign);
    m.off_logits = sc; sc = align_up(sc + (size_t)cap->max_seqs * c->vocab * 4, kAlign);
    m.off_rope = sc; sc = align_up(sc + (size_t)P.ctx_stride * (c->head_dim / 2) * 8, kAlign);
    m.packed_bytes = 0;
    for (const auto& nk : packed_shapes(c))
      if (packs(c, nk.first, nk.second)) m.packed_bytes += align_up(packed_weight_bytes(nk.first, nk.second), kAlign);
    m.off_packed = sc; sc = align_up(sc + m.packed_bytes, kAlign);
  }
  P.kv_bytes = kv;
  const size_t S = (size_t)cap->max_seqs;
  P.off_state = sc; sc = align_up(sc + 6 * S * 4, kAlign);
  P.off_seq_slot = sc; sc = align_up(sc + S * 4, kAlign);
  P.off_rows = sc; sc = align_up(sc + 5 * (size_t)cap->max_prefill_tokens * 4, kAlign);
  P.off_prompt = sc; sc = align_up(sc + 4 * S * 4, kAlign);
  P.off_err = sc; sc = align_up(sc + 4, kAlign);
  P.off_partials = sc; sc = align_up(sc + S * P.n_chunks * 5 * 4, kAlign);
  P.off_count = sc; sc = align_up(sc + 4, kAlign);
  P.off_act = sc; sc = align_up(sc + S * 4, kAlign);
  P.off_drows = sc; sc = align_up(sc + 4 * S * 4, kAlign);
  P.off_pfx = sc; sc = align_up(sc + 2 * S * 4, kAlign);
  P.off_score = sc; sc = align_up(sc + S * P.n_chunks * 6 * 4, kAlign);
  P.fused = sen->vocab % 4 == 0;
  for (int i = 0; i < P.nm; ++i) P.fused = P.fused && packs(cf[i], cf[i]->vocab, cf[i]->d_model);
  P.noise_rows = P.fused ? (int)std::min<size_t>(S, kStreamMaxRows) : 0;
  const size_t NR = (size_t)P.noise_rows;
  P.off_noise = sc; sc = align_up(sc + NR * sen->vocab * 4, kAlign);
  P.off_part_sen = sc; sc = align_up(sc + NR * kSampleParts * 5 * 4, kAlign);
  P.off_part_jun = sc; sc = align_up(sc + (P.nm == 2 ? NR : 0) * kSampleParts * 5 * 4, kAlign);
  P.scratch_bytes = sc;
  return P;
}

}  // namespace

struct tandem_handle {
  Model m[2];                 // 0: senior, 1: junior (unused when nm == 1)
  int nm = 2;                 // 1: a single-model rollout of the senior (no junior)
  Plan plan;
  tandem_switch_cfg sw;
  tandem_sample_cfg smp;
  tandem_capacity cap;
  tandem_outputs out;
  unsigned long long thr;
  uint32_t key0, key1;
  hipStream_t stream;
  // The two models' forwards are independent until sampling: the junior's
  // runs on a second stream forked from and joined back into `stream`.
  hipStream_t side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  // one event per layer of each model, recorded after that layer's FFN-input
  // norm (the two streams' attentions take turns, see forward_pair)
  std::vector<hipEvent_t> ev_att[2];
  // Step graphs are captured on a stream of the library's own (the caller's
  // may be the legacy null stream, which cannot be captured) and replayed on
  // the caller's stream.
  hipStream_t gstream = nullptr;
  int n_cu = 256;             // compute units of the device (split-K sizing)
  int32_t *owner, *c, *t, *pos, *pending, *done;
  int32_t* seq_slot;
  int32_t *row_slot, *row_pos, *row_tok;                // prompt rows of one prefill chunk
  int32_t *grp_row0, *grp_n;                            // their 16-row groups (attention)
  // Decode rows: row r carries sequence act[r].  After a prefill act is the
  // identity; with EOS on, a stable partition (unfinished first) runs every
  // kCompactEvery steps and the launched row count shrinks to the smallest
  // multiple of kCompactBucket that covers the unfinished sequences.
  int32_t* act;
  int32_t *drow_tok, *drow_slot, *drow_pos, *drow_done;
  int R_launch = 0;
  // Shared prompt prefix.  The G sequences of a prompt hold the same K/V at
  // the prompt positions: decode attention reads positions [0, lo) (lo = the
  // prompt length - 1 rounded down to 16) from the slot of the prompt's first
  // sequence and each row's own slot from lo on.  The per-row tables (lo,
  // prefix slot) follow the act order (rebuilt at prefill and at each
  // compaction).
  bool share = false;
  int32_t *row_lo, *pfx_slot;
  int G = 1;
  int steps_since_compact = 0;
  int32_t *p_end, *p_len, *p_rbase, *p_gbase;         // per prompt (device)
  // A prompt token id outside [0, vocab) sets this device flag (and is read
  // as 0); it is reported at the next call that synchronises.
  int32_t* d_err;
  // Pinned host staging of the per-prompt table; the next prefill refills it
  // only once the previous upload has left it (ev_stage).
  int32_t* h_stage = nullptr;
  hipEvent_t ev_stage = nullptr;
  float* partials;
  // Sampling inside the LM heads (see Plan::fused): noise and partials, the
  // event that orders the noise before the senior's LM head, and whether the
  // last step sampled this way (its logits were then never stored)
  bool fused = false;
  float *noise = nullptr, *part_sen = nullptr, *part_jun = nullptr;
  hipEvent_t ev_noise = nullptr;
  bool last_fused = false;
  int32_t* d_count;
  int32_t* h_sync = nullptr;  // pinned: [0] a count read back, [1] the error flag
  int n_seq = 0;
  bool prefilled = false;
  bool stepped = false;       // a step has run since the last prefill (its logits are in place)
  float* score_part = nullptr;  // partials of tandem_score_step
  bool poisoned = false;
  std::string err = "no error";
  // instrumentation: event pairs per kernel class
  int timing = 0;             // class mask and flags
  std::vector<hipEvent_t> ev_pool;                   // eager launches
  size_t ev_used = 0;
  std::vector<std::pair<int, size_t>> ev_marks;      // (class, index of the begin event), not yet summed
  double acc_ms[TANDEM_K_CLASSES] = {};
  int64_t acc_n[TANDEM_K_CLASSES] = {};
  // Decode steps replay a captured HIP graph of the whole step (both
  // forwards, sampling, handoff rule); rebuilt when the batch or the schedule
  // flags change.  (Event records captured into a graph do not carry launch
  // times, so timed steps are launched eagerly.)
  hipGraphExec_t graph = nullptr;
  int graph_R = -1, graph_flags = -1;
};

namespace {

// Record a begin event for a kernel class on stream st (no-op unless timing
// is enabled).
hipError_t tim_begin(tandem_handle* h, int klass, size_t* idx, hipStream_t st) {
  *idx = SIZE_MAX;
  if (!(h->timing & (1 << klass))) return hipSuccess;
  while (h->ev_pool.size() < h->ev_used + 2) {
    hipEvent_t e;
    hipError_t r = hipEventCreate(&e);
    if (r != hipSuccess) return r;
    h->ev_pool.push_back(e);
  }
  *idx = h->ev_used;
  h->ev_used += 2;
  h->ev_marks.push_back({klass, *idx});
  return hipEventRecord(h->ev_pool[*idx], st);
}
hipError_t tim_end(tandem_handle* h, size_t idx, hipStream_t st) {
  if (idx == SIZE_MAX) return hipSuccess;
  return hipEventRecord(h->ev_pool[idx + 1], st);
}

// Add the recorded launch times to the class sums.
hipError_t harvest_all(tandem_handle* h) {
  if (h->ev_marks.empty()) return hipSuccess;
  hipError_t r = hipStreamSynchronize(h->stream);
  if (r != hipSuccess) return r;
  for (const auto& mk : h->ev_marks) {
    float ms = 0.f;
    r = hipEventElapsedTime(&ms, h->ev_pool[mk.second], h->ev_pool[mk.second + 1]);
    if (r != hipSuccess) return r;
    h->acc_ms[mk.first] += ms;
    h->acc_n[mk.first] += 1;
  }
  h->ev_marks.clear();
  h->ev_used = 0;
  return hipSuccess;
}

void drop_graphs(tandem_handle* h) {
  if (h->graph) (void)hipGraphExecDestroy(h->graph);
  h->graph = nullptr;
  h->graph_R = -1;
  h->graph_flags = -1;
}

}  // namespace

// Launch one kernel class between timing events on the launch stream `st`.
#define TIMED(klass, expr)                                                                 \
  do {                                                                                     \
    size_t ti_ = 0;                                                                        \
    HIPCHK(tim_begin(h, (klass), &ti_, st));                                               \
    HIPCHK(expr);                                                                          \
    HIPCHK(tim_end(h, ti_, st));                                                           \
  } while (0)

#define HIPCHK(expr)                                                                       \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess) {                                                                \
      h->poisoned = true;                                                                  \
      return fail(&h->err, TANDEM_E_HIP, std::string("HIP error in ") + #expr + ": " +     \
                                             hipGetErrorString(e_));                       \
    }                                                                                      \
  } while (0)

namespace {

// Split-K slices of one projection: as many as keep (tiles x slices) within
// one workgroup per compute unit (more slices than that leave a straggling
// second round), at most kSplitMax, one 64-wide k chunk each at least, and
// what the partial-sum workspace holds.
int choose_splits(int M, int N, int K, size_t ws_floats, int n_cu) {
  const int m_tiles = (M + 127) / 128, n_tiles = (N + 127) / 128;
  const int base = m_tiles * n_tiles;
  int S = n_cu / base;
  if (S > kSplitMax) S = kSplitMax;
  if (S > K / 64) S = K / 64;
  const size_t cap_ws = ws_floats / ((size_t)M * N);
  if ((size_t)S > cap_ws) S = (int)cap_ws;
  if (S < 1) S = 1;
  return S;
}

// One projection out = A . W^T (M rows): the streaming kernel over the packed
// copy for decode-sized M, the tiled kernel otherwise.  EPI_PARTIAL writes
// split-K partial tiles (stride M * N floats) and returns their count in *S;
// EPI_STORE writes out[m * N + n].
// A16: the activations are fp16 rows and Wp an fp16 packed copy (only on the
// streaming path, which the caller's choice of format has already implied).
tandem_status gemm(tandem_handle* h, const Model& m, const void* A, const void* W, const void* Wp, int M, int N,
                   int K, int epi, float* out, int* S, hipStream_t st, bool a16 = false) {
  const int dt = m.cfg.weight_dtype == TANDEM_BF16 ? DT_BF16 : DT_F32;
  *S = 1;
  if (Wp && M <= kStreamMaxRows) {
    const StreamPlan pl = plan_stream_gemm(M, N, K, h->n_cu, m.p.ws_floats, epi == EPI_STORE ? kPlanStore : kPlanPartial);
    GemmStreamArgs a{};
    a.A = A; a.Wp = Wp; a.M = M; a.N = N; a.K = K; a.a16 = a16; a.epi = epi; a.out = out; a.ldo = N;
    a.split_stride = (long)M * N;
    a.nbw = pl.nbw; a.S = pl.S; a.cps = pl.cps; a.n_groups = pl.n_groups; a.grid = pl.grid;
    *S = pl.S;
    TIMED(TANDEM_K_GEMM, launch_gemm_stream(a, st));
    return TANDEM_OK;
  }
  GemmArgs g{};
  g.dt = dt; g.A = A; g.W = W; g.M = M; g.N = N; g.K = K; g.epi = epi;
  g.Wp = Wp; g.a16 = a16;                  // prefill-sized products read the packed copy too
  g.out = out; g.ldo = N; g.split_stride = (long)M * N;
  g.splits = epi == EPI_PARTIAL ? choose_splits(M, N, K, m.p.ws_floats, h->n_cu) : 1;
  TIMED(TANDEM_K_GEMM, launch_gemm(g, S, st));
  return TANDEM_OK;
}

// Gate/up projection and SwiGLU: x_f = silu(A W_g^T) * (A W_u^T) in split
// format.  Decode-sized M streams the pair-interleaved packed copy, with the
// SwiGLU in the GEMM epilogue (one K slice) or in a pass over the split-K
// partials; larger M uses the tiled kernel.
tandem_status gate_up(tandem_handle* h, const Model& m, const Layer& L, int M, hipStream_t st) {
  const tandem_model_cfg& c = m.cfg;
  const int dt = c.weight_dtype == TANDEM_BF16 ? DT_BF16 : DT_F32;
  const int d = c.d_model, F = c.ffn_dim;
  if (L.p_gate_up && M <= kStreamMaxRows) {
    const StreamPlan pl = plan_stream_gemm(M, 2 * F, d, h->n_cu, m.p.ws_floats, kPlanSwiglu);
    GemmStreamArgs a{};
    a.A = m.xa; a.Wp = L.p_gate_up; a.M = M; a.N = 2 * F; a.K = d; a.a16 = m.ffn16;
    a.nbw = pl.nbw; a.S = pl.S; a.cps = pl.cps; a.n_groups = pl.n_groups; a.grid = pl.grid;
    if (pl.S == 1) {
      a.epi = EPI_SWIGLU; a.out = (float*)m.xf; a.ldo = F;
      TIMED(TANDEM_K_GEMM, launch_gemm_stream(a, st));
    } else {
      a.epi = EPI_PARTIAL; a.out = m.ws; a.ldo = 2 * F; a.split_stride = (long)M * 2 * F;
      TIMED(TANDEM_K_GEMM, launch_gemm_stream(a, st));
      TIMED(TANDEM_K_OTHER, launch_swiglu_finish(m.ws, pl.S, (long)M * 2 * F, M, F, true, m.ffn16, m.xf, st));
    }
    return TANDEM_OK;
  }
  // prefill-sized: the tiled GEMM on the packed (pair-interleaved) copy when
  // there is one, fp16 activations with it (the partial columns then follow
  // the interleaved order)
  int S = 1;
  const bool pk = L.p_gate_up != nullptr && M > 64;
  const bool a16 = pk && m.ffn16;
  if (split_gate_up(&c)) {
    GemmArgs g{};
    g.dt = dt; g.A = m.xa; g.W = L.w_gate_up; g.M = M; g.N = 2 * F; g.K = d; g.epi = EPI_PARTIAL;
    g.Wp = pk ? L.p_gate_up : nullptr; g.a16 = a16;
    g.out = m.ws; g.ldo = 2 * F; g.split_stride = (long)M * 2 * F;
    g.splits = choose_splits(M, 2 * F, d, m.p.ws_floats, h->n_cu);
    TIMED(TANDEM_K_GEMM, launch_gemm(g, &S, st));
    TIMED(TANDEM_K_OTHER, launch_swiglu_finish(m.ws, S, (long)M * 2 * F, M, F, pk, a16, m.xf, st));
    return TANDEM_OK;
  }
  GemmArgs g{};
  g.dt = dt; g.A = m.xa; g.W = L.w_gate_up; g.M = M; g.N = F; g.K = d; g.epi = EPI_SWIGLU;
  g.Wp = pk ? L.p_gate_up : nullptr; g.a16 = a16;
  g.out = (float*)m.xf; g.ldo = F; g.splits = 1;
  TIMED(TANDEM_K_GEMM, launch_gemm(g, &S, st));
  return TANDEM_OK;
}

#define CALL(expr)                                                                         \
  do {                                                                                     \
    tandem_status s_ = (expr);                                                             \
    if (s_ != TANDEM_OK) return s_;                                                        \
  } while (0)

// Forward R rows through one model.  Rows read their token, cache slot and
// position from the row arrays; done rows (row_done != NULL) skip the cache
// append and produce zero attention.  With lm_head the logits land in m.logits.
// One model's decode/prefill forward in three pieces: embedding + first norm,
// one layer, final LM head.
struct FwdRows {
  int R;
  const int32_t *tok, *slot, *pos, *done;
  // prompt rows: groups of at most 16 consecutive rows of one prompt (the
  // attention's row blocks); NULL at decode
  const int32_t *grp_row0 = nullptr, *grp_n = nullptr;
  int n_groups = 0;
  bool shared_prefix = false;   // decode rows reading the prompt prefix through the prefix tables
};

tandem_status forward_embed(tandem_handle* h, Model& m, const FwdRows& fr, hipStream_t st) {
  const tandem_model_cfg& c = m.cfg;
  const int dt = c.weight_dtype == TANDEM_BF16 ? DT_BF16 : DT_F32;
  TIMED(TANDEM_K_OTHER, launch_embed_norm(dt, fr.tok, m.embed, c.d_model, m.layers[0].attn_norm, c.rms_eps, m.h,
                                          m.xa, fr.R, st));
  return TANDEM_OK;
}

// att_wait: an event the layer's attention waits for first (NULL: none);
// att_done: recorded after the FFN-input norm launch (NULL: none).
tandem_status forward_layer(tandem_handle* h, Model& m, int l, const FwdRows& fr, hipStream_t st,
                            hipEvent_t att_wait = nullptr, hipEvent_t att_done = nullptr) {
  const tandem_model_cfg& c = m.cfg;
  const int dt = c.weight_dtype == TANDEM_BF16 ? DT_BF16 : DT_F32;
  const int d = c.d_model, hd = c.head_dim, nq = c.n_q_heads, nkv = c.n_kv_heads;
  const int qkv = m.p.qkv_dim, att = m.p.att_dim;
  const int R = fr.R;
  const Layer& L = m.layers[l];
  CacheGeom cg;
  cg.k = m.kc + (size_t)l * m.layer_stride * m.p.esz;
  cg.v = m.vc + (size_t)l * m.layer_stride * m.p.esz;
  cg.ctx_stride = h->plan.ctx_stride;
  cg.slot_stride = m.slot_stride;

  int S = 1;
  CALL(gemm(h, m, m.xa, L.w_qkv, L.p_qkv, R, qkv, d, EPI_PARTIAL, m.ws, &S, st));

  {
    QkvPostArgs qp{};
    qp.dt = dt; qp.ws = m.ws; qp.S = S; qp.ws_stride = (long)R * qkv;
    qp.R = R; qp.nq = nq; qp.nkv = nkv; qp.hd = hd;
    qp.q_norm = c.qk_norm ? L.q_norm : nullptr; qp.k_norm = c.qk_norm ? L.k_norm : nullptr;
    qp.eps = c.rms_eps; qp.rope = m.rope;
    qp.row_slot = fr.slot; qp.row_pos = fr.pos; qp.row_done = fr.done;
    qp.q_out = m.q; qp.cache = cg;
    TIMED(TANDEM_K_OTHER, launch_qkv_post(qp, st));
  }

  AttnArgs aa{};
  aa.dt = dt; aa.q = m.q; aa.R = R; aa.nq = nq; aa.nkv = nkv; aa.hd = hd; aa.cache = cg;
  aa.row_slot = fr.slot; aa.row_pos = fr.pos; aa.row_done = fr.done; aa.out = m.xa;
  aa.grp_row0 = fr.grp_row0; aa.grp_n = fr.grp_n; aa.n_groups = fr.n_groups;
  if (fr.shared_prefix) {
    aa.row_lo = h->row_lo; aa.pfx_slot = h->pfx_slot;
  }
  if (att_wait) HIPCHK(hipStreamWaitEvent(st, att_wait, 0));
  TIMED(TANDEM_K_ATTENTION, launch_attention(aa, st));

  // the FFN's activations are fp16 when both its products have fp16 packed
  // copies (the streaming GEMM up to 128 rows, the tiled one above; the
  // output of the last layer's norm feeds the LM head only)
  const bool f16 = m.ffn16;
  const bool last = l + 1 == c.n_layers;
  CALL(gemm(h, m, m.xa, L.w_o, L.p_o, R, d, att, EPI_PARTIAL, m.ws, &S, st));
  TIMED(TANDEM_K_OTHER, launch_resid_norm(dt, m.ws, S, (long)R * d, m.h, L.ffn_norm, c.rms_eps, m.xa, R, d, f16, st));
  // the other model's next attention may start (see forward_pair)
  if (att_done) HIPCHK(hipEventRecord(att_done, st));

  CALL(gate_up(h, m, L, R, st));
  CALL(gemm(h, m, m.xf, L.w_down, L.p_down, R, d, c.ffn_dim, EPI_PARTIAL, m.ws, &S, st, f16));
  const float* next_gain = last ? m.final_norm : m.layers[l + 1].attn_norm;
  const bool next16 = last && m.lm16;
  TIMED(TANDEM_K_OTHER, launch_resid_norm(dt, m.ws, S, (long)R * d, m.h, next_gain, c.rms_eps, m.xa, R, d, next16, st));
  return TANDEM_OK;
}

// The LM head's launch plan on the streaming GEMM (one K slice, plain or
// sampling epilogue); its grid is the number of sampling partials per row.
StreamPlan head_plan(const tandem_handle* h, const Model& m, int R) {
  return plan_stream_gemm(R, m.cfg.vocab, m.cfg.d_model, h->n_cu, m.p.ws_floats, kPlanStore);
}

// The LM head of model i (0 senior, 1 junior): logits [R][V], or, when the
// step samples inside the LM heads, per-row sampling partials (the senior's
// head waits for the step's noise, ev_noise, when that was launched on
// another stream).
tandem_status forward_head(tandem_handle* h, int i, const FwdRows& fr, bool fused, hipStream_t st,
                           hipEvent_t wait_noise = nullptr) {
  Model& m = h->m[i];
  const tandem_model_cfg& c = m.cfg;
  int S = 1;
  if (!fused) {
    CALL(gemm(h, m, m.xa, m.lm_head, m.p_lm, fr.R, c.vocab, c.d_model, EPI_STORE, m.logits, &S, st, m.lm16));
    return TANDEM_OK;
  }
  if (wait_noise) HIPCHK(hipStreamWaitEvent(st, wait_noise, 0));
  const StreamPlan pl = head_plan(h, m, fr.R);
  GemmStreamArgs a{};
  a.A = m.xa; a.Wp = m.p_lm; a.M = fr.R; a.N = c.vocab; a.K = c.d_model; a.a16 = true; a.epi = EPI_SAMPLE;
  a.ldo = c.vocab;
  a.nbw = pl.nbw; a.S = pl.S; a.cps = pl.cps; a.n_groups = pl.n_groups; a.grid = pl.grid;
  SampleEpiArgs& sm = a.smp;
  sm.noise = h->noise; sm.act = h->act; sm.owner = h->owner; sm.done = h->done;
  sm.model = i == 0 ? 1 : 0;
  sm.temp = h->smp.temperature; sm.eos_id = h->smp.eos_id;
  sm.eos_bias = i == 0 ? h->smp.eos_bias_senior : h->smp.eos_bias_junior;
  sm.part = i == 0 ? h->part_sen : h->part_jun;
  sm.n_part = pl.grid;
  TIMED(TANDEM_K_GEMM, launch_gemm_stream(a, st));
  return TANDEM_OK;
}

// This step's Gumbel noise for the sampling inside the LM heads.
tandem_status launch_noise(tandem_handle* h, int R, hipStream_t st) {
  TIMED(TANDEM_K_SAMPLE, launch_gumbel_noise(h->act, h->t, h->done, R, h->m[0].cfg.vocab, h->key0, h->key1,
                                             h->noise, st));
  return TANDEM_OK;
}

tandem_status forward(tandem_handle* h, int i, const FwdRows& fr, bool lm_head, bool fused, hipStream_t st) {
  Model& m = h->m[i];
  CALL(forward_embed(h, m, fr, st));
  for (int l = 0; l < m.cfg.n_layers; ++l) CALL(forward_layer(h, m, l, fr, st));
  if (lm_head) CALL(forward_head(h, i, fr, fused, st));
  return TANDEM_OK;
}

// Both models' forwards over the same rows: the junior on the side stream,
// the senior on the main stream, joined before anything that reads either.
// The two models' decode attentions are bound by HBM bandwidth, their
// projections mostly by latency: the step runs both forwards on two streams
// and lets the attention launches take turns, so each model's attention runs
// beside the other model's projections rather than beside its attention.
// The turn order interleaves the layers evenly (layer l of a model with L
// layers at (l + 1/2) / L); an attention waits until the layer before it in
// that order, of the other model, has run its attention, O projection and
// FFN-input norm: those two kernels of the senior, on its critical path, are
// then not slowed by the junior's attention grid beside them (the O
// projection and norm of a model take about 25 us alone and 80 us beside the
// other model's attention).
//
// With the sampling inside the LM heads (fused), the step's Gumbel noise is
// generated first on the junior's stream (whose chain is the shorter one) and
// the senior's LM head waits for it.
tandem_status forward_pair(tandem_handle* h, const FwdRows& fr, bool lm_head, bool fused = false) {
  hipStream_t st = h->stream;
  if (h->nm == 1 || (h->timing & TANDEM_TIMING_SERIAL)) {
    if (fused) CALL(launch_noise(h, fr.R, st));
    for (int i = 0; i < h->nm; ++i) CALL(forward(h, i, fr, lm_head, fused, st));
    return TANDEM_OK;
  }
  HIPCHK(hipEventRecord(h->ev_fork, st));
  HIPCHK(hipStreamWaitEvent(h->side, h->ev_fork, 0));
  hipStream_t sts[2] = {st, h->side};
  if (fused) {
    CALL(launch_noise(h, fr.R, sts[1]));
    HIPCHK(hipEventRecord(h->ev_noise, sts[1]));
  }
  Model* ms[2] = {&h->m[0], &h->m[1]};
  {
    const int L[2] = {ms[0]->cfg.n_layers, ms[1]->cfg.n_layers};
    CALL(forward_embed(h, *ms[0], fr, sts[0]));
    CALL(forward_embed(h, *ms[1], fr, sts[1]));
    int next[2] = {0, 0}, prev_model = -1, prev_layer = -1;
    while (next[0] < L[0] || next[1] < L[1]) {
      // the model whose next layer comes first in the interleaved order
      int i;
      if (next[0] >= L[0]) i = 1;
      else if (next[1] >= L[1]) i = 0;
      else i = (2 * next[0] + 1) * (long)L[1] <= (2 * next[1] + 1) * (long)L[0] ? 0 : 1;
      const int l = next[i]++;
      hipEvent_t wait = (prev_model >= 0 && prev_model != i) ? h->ev_att[prev_model][prev_layer] : nullptr;
      CALL(forward_layer(h, *ms[i], l, fr, sts[i], wait, h->ev_att[i][l]));
      prev_model = i;
      prev_layer = l;
    }
    if (lm_head) {
      CALL(forward_head(h, 1, fr, fused, sts[1]));
      CALL(forward_head(h, 0, fr, fused, sts[0], fused ? h->ev_noise : nullptr));
    }
  }
  HIPCHK(hipEventRecord(h->ev_join, h->side));
  HIPCHK(hipStreamWaitEvent(st, h->ev_join, 0));
  return TANDEM_OK;
}

// Enqueue one decode step (both forwards, sampling, outputs, handoff rule).
// fused: sample inside the LM heads (no logits stored; see step_fused).
tandem_status record_step(tandem_handle* h, const int32_t* forced, const tandem_debug* dbg, bool fused) {
  const int R = h->R_launch;
  hipStream_t st = h->stream;
  {
    GatherRowsArgs ga{};
    ga.act = h->act; ga.R = R;
    ga.pending = h->pending; ga.seq_slot = h->seq_slot; ga.pos = h->pos; ga.done = h->done;
    ga.row_tok = h->drow_tok; ga.row_slot = h->drow_slot; ga.row_pos = h->drow_pos; ga.row_done = h->drow_done;
    TIMED(TANDEM_K_OTHER, launch_gather_rows(ga, st));
    FwdRows fr{R, h->drow_tok, h->drow_slot, h->drow_pos, h->drow_done};
    fr.shared_prefix = h->share;
    tandem_status s = forward_pair(h, fr, true, fused);
    if (s != TANDEM_OK) return s;
  }
  const int V = h->m[0].cfg.vocab;
  FinishArgs fa{};
  if (fused) {
    fa.part_sen = h->part_sen; fa.n_sen = head_plan(h, h->m[0], R).grid;
    fa.part_jun = h->part_jun; fa.n_jun = head_plan(h, h->m[h->nm - 1], R).grid;
    fa.x_sen = (const uint16_t*)h->m[0].xa; fa.w_lm = (const uint16_t*)h->m[0].lm_head; fa.d = h->m[0].cfg.d_model;
  } else {
    SampleArgs sa{};
    sa.z_sen = h->m[0].logits; sa.z_jun = h->m[h->nm - 1].logits; sa.R = R; sa.V = V;
    sa.temp = h->smp.temperature; sa.eos_id = h->smp.eos_id;
    sa.eos_bias_sen = h->smp.eos_bias_senior; sa.eos_bias_jun = h->smp.eos_bias_junior;
    sa.key0 = h->key0; sa.key1 = h->key1;
    sa.owner = h->owner; sa.t = h->t; sa.done = h->done; sa.act = h->act;
    sa.partials = h->partials; sa.chunk = kVocabChunk;
    TIMED(TANDEM_K_SAMPLE, launch_sample_partials(sa, h->plan.n_chunks, st));
    if (dbg) {
      if (dbg->logits_senior) HIPCHK(launch_scatter_rows(h->m[0].logits, h->act, R, V, dbg->logits_senior, st));
      if (dbg->logits_junior && h->nm == 2)
        HIPCHK(launch_scatter_rows(h->m[1].logits, h->act, R, V, dbg->logits_junior, st));
    }
  }
  fa.z_sen = h->m[0].logits; fa.R = R; fa.V = V; fa.act = h->act;
  fa.temp = h->smp.temperature; fa.eos_id = h->smp.eos_id; fa.eos_bias_sen = h->smp.eos_bias_senior;
  fa.partials = h->partials; fa.n_chunks = h->plan.n_chunks;
  fa.forced = forced;
  fa.key0 = h->key0; fa.key1 = h->key1; fa.thr = h->thr; fa.mode = h->sw.mode; fa.cap_k = h->sw.cap_k;
  fa.bnd = h->sw.boundary_bits; fa.max_new = h->smp.max_new_tokens;
  fa.owner = h->owner; fa.c = h->c; fa.t = h->t; fa.pos = h->pos; fa.pending = h->pending; fa.done = h->done;
  fa.out_tok = h->out.tokens; fa.out_own = h->out.owner; fa.out_lp = h->out.senior_logprob;
  fa.out_len = h->out.length; fa.ld_out = h->smp.max_new_tokens;
  fa.dbg_sampled = dbg ? dbg->sampled : nullptr; fa.dbg_margin = dbg ? dbg->margin : nullptr;
  TIMED(TANDEM_K_SAMPLE, launch_sample_finish(fa, st));
  return TANDEM_OK;
}

// Shared-prefix tables of the launched decode rows in the current act order
// (see tandem_handle::share), built on the device.
tandem_status prefix_tables(tandem_handle* h) {
  if (!h->share) return TANDEM_OK;
  HIPCHK(launch_prefix_rows(h->act, h->R_launch, h->G, h->p_len, h->row_lo, h->pfx_slot, h->stream));
  return TANDEM_OK;
}

// After a synchronisation that read the error flag into h_sync[1]: a prompt
// token id of the current batch was outside the vocabulary.
tandem_status batch_error(tandem_handle* h) {
  if (!h->h_sync[1]) return TANDEM_OK;
  h->prefilled = false;
  return fail(&h->err, TANDEM_E_ARG,
              "a prompt token id passed to tandem_prefill was outside [0, vocab): the batch ran with token 0 in its "
              "place and is void; prefill again");
}

// Read the batch's error flag along with a count already on its way to
// h_sync[0], then synchronise the stream.
tandem_status sync_read(tandem_handle* h, const int32_t* d_count) {
  hipStream_t st = h->stream;
  if (d_count) HIPCHK(hipMemcpyAsync(h->h_sync, d_count, 4, hipMemcpyDeviceToHost, st));
  HIPCHK(hipMemcpyAsync(h->h_sync + 1, h->d_err, 4, hipMemcpyDeviceToHost, st));
  HIPCHK(hipStreamSynchronize(st));
  return batch_error(h);
}

// With EOS on, sequences finish at different steps: every kCompactEvery steps
// partition the batch (unfinished sequences first, stable) and shrink the
// launched row count.  One host synchronisation per compaction (the launched
// row count is a host value).
tandem_status maybe_compact(tandem_handle* h) {
  if (h->smp.eos_id < 0 || ++h->steps_since_compact < kCompactEvery) return TANDEM_OK;
  h->steps_since_compact = 0;
  HIPCHK(launch_compact(h->done, h->n_seq, h->act, h->d_count, h->stream));
  CALL(sync_read(h, h->d_count));
  const int n_act = h->h_sync[0];
  int R = (std::max(n_act, 1) + kCompactBucket - 1) / kCompactBucket * kCompactBucket;
  if (R > h->n_seq) R = h->n_seq;
  if (R < h->R_launch) {
    h->R_launch = R;
    drop_graphs(h);                   // captured for the old row count
  }
  return prefix_tables(h);            // the act order changed
}

// Whether a step samples inside the LM heads: the handle's models allow it,
// the launched rows fit one streaming tile, the caller asked for no logits and
// has not switched the fusion off (TANDEM_TIMING_SEPARATE_SAMPLE).
bool step_fused(const tandem_handle* h, const tandem_debug* dbg) {
  return h->fused && h->R_launch <= h->plan.noise_rows && !(h->timing & TANDEM_TIMING_SEPARATE_SAMPLE) &&
         !(dbg && (dbg->logits_senior || dbg->logits_junior));
}

// Capture the step into h->graph (the streams return to normal operation
// whatever happens inside).
tandem_status capture_step(tandem_handle* h) {
  hipStream_t caller = h->stream;
  HIPCHK(hipStreamBeginCapture(h->gstream, hipStreamCaptureModeThreadLocal));
  h->stream = h->gstream;                 // the step's main stream while recording
  tandem_status s = record_step(h, nullptr, nullptr, step_fused(h, nullptr));
  h->stream = caller;
  hipGraph_t graph = nullptr;
  hipError_t e = hipStreamEndCapture(h->gstream, &graph);
  if (s != TANDEM_OK) {
    if (graph) (void)hipGraphDestroy(graph);
    return s;
  }
  HIPCHK(e);
  e = hipGraphInstantiate(&h->graph, graph, nullptr, nullptr, 0);
  (void)hipGraphDestroy(graph);
  if (e != hipSuccess) h->graph = nullptr;
  HIPCHK(e);
  return TANDEM_OK;
}

tandem_status step_impl(tandem_handle* h, const int32_t* forced, const tandem_debug* dbg, int32_t* n_active) {
  if (!h) return fail(nullptr, TANDEM_E_ARG, "handle is NULL");
  if (h->poisoned) return fail(&h->err, TANDEM_E_STATE, "handle is poisoned by an earlier HIP error");
  if (!h->prefilled) return fail(&h->err, TANDEM_E_STATE, "tandem_step before tandem_prefill");
  {
    tandem_status s = maybe_compact(h);
    if (s != TANDEM_OK) return s;
  }
  const int R = h->R_launch;
  hipStream_t st = h->stream;
  const bool timed = (h->timing & ((1 << TANDEM_K_CLASSES) - 1)) != 0;
  const bool graph = !forced && !dbg && !timed && !(h->timing & TANDEM_TIMING_EAGER);
  if (graph) {
    if (!h->graph || h->graph_R != R || h->graph_flags != h->timing) {
      drop_graphs(h);
      tandem_status s = capture_step(h);
      if (s != TANDEM_OK) {
        drop_graphs(h);
        return s;
      }
      h->graph_R = R;
      h->graph_flags = h->timing;
    }
    // replayed on the caller's stream itself (a graph captured on one stream
    // may be launched on any): ordering it through the capture stream with an
    // event pair per step cost about 0.15 ms per step
    HIPCHK(hipGraphLaunch(h->graph, st));
  } else {
    tandem_status s = record_step(h, forced, dbg, step_fused(h, dbg));
    if (s != TANDEM_OK) return s;
  }
  h->stepped = true;
  h->last_fused = step_fused(h, dbg);
  if (n_active) {
    HIPCHK(launch_count_active(h->done, h->n_seq, h->d_count, st));
    CALL(sync_read(h, h->d_count));
    *n_active = h->h_sync[0];
  }
  return TANDEM_OK;
}

}  // namespace

namespace {
tandem_status grpo_check(const tandem_grpo_cfg* c, size_t* bytes, GrpoArgs* a) {
  if (!c) return fail(nullptr, TANDEM_E_ARG, "tandem_grpo: cfg is NULL");
  if (c->n_groups < 1 || c->group_size < 1 || c->max_new_tokens < 1)
    return fail(nullptr, TANDEM_E_SHAPE, "tandem_grpo: n_groups, group_size and max_new_tokens must be >= 1");
  const long long S = (long long)c->n_groups * c->group_size;
  if (S * c->max_new_tokens >= (1LL << 24))
    return fail(nullptr, TANDEM_E_SHAPE, "tandem_grpo: S * max_new_tokens must be below 2^24");
  if (!(c->clip_eps >= 0.f && c->clip_eps < 1.f))
    return fail(nullptr, TANDEM_E_ARG, "tandem_grpo: clip_eps must lie in [0, 1)");
  a->S = (int)S; a->G = c->group_size; a->T = c->max_new_tokens; a->eps = c->clip_eps;
  a->n_chunks = (a->T + kGrpoChunk - 1) / kGrpoChunk;
  // counts [S] int32, partial sums [S][n_chunks] float, a ticket int32, each 256-aligned
  const size_t cnt_b = ((size_t)S * 4 + 255) / 256 * 256;
  *bytes = cnt_b + ((size_t)S * a->n_chunks * 4 + 255) / 256 * 256 + 256;
  return TANDEM_OK;
}
}  // namespace

extern "C" {

const char* tandem_status_string(tandem_status s) {
  switch (s) {
    case TANDEM_OK: return "TANDEM_OK";
    case TANDEM_E_ARG: return "TANDEM_E_ARG";
    case TANDEM_E_SHAPE: return "TANDEM_E_SHAPE";
    case TANDEM_E_CAPACITY: return "TANDEM_E_CAPACITY";
    case TANDEM_E_STATE: return "TANDEM_E_STATE";
    case TANDEM_E_HIP: return "TANDEM_E_HIP";
    case TANDEM_E_UNSUPPORTED: return "TANDEM_E_UNSUPPORTED";
  }
  return "TANDEM_E_UNKNOWN";
}

const char* tandem_last_error(const tandem_handle* h) { return h ? h->err.c_str() : g_err.c_str(); }

tandem_status tandem_workspace_size(const tandem_model_cfg* senior, const tandem_model_cfg* junior,
                                    const tandem_capacity* cap, size_t* kv_bytes, size_t* scratch_bytes) {
  if (!senior || !cap || !kv_bytes || !scratch_bytes)
    return fail(nullptr, TANDEM_E_ARG, "tandem_workspace_size: NULL argument");
  tandem_status s;
  if ((s = check_cfg(senior, "senior", nullptr)) != TANDEM_OK) return s;
  if (junior && (s = check_cfg(junior, "junior", nullptr)) != TANDEM_OK) return s;
  if (junior && senior->vocab != junior->vocab)
    return fail(nullptr, TANDEM_E_SHAPE, "senior and junior must share one vocabulary");
  if ((s = check_cap(cap, nullptr)) != TANDEM_OK) return s;
  Plan P = make_plan(senior, junior, cap);
  *kv_bytes = P.kv_bytes;
  *scratch_bytes = P.scratch_bytes;
  return TANDEM_OK;
}

tandem_status tandem_init(const tandem_model* senior, const tandem_model* junior, const tandem_switch_cfg* sw,
                          const tandem_sample_cfg* smp, const tandem_capacity* cap, void* kv_arena,
                          size_t kv_bytes, void* scratch, size_t scratch_bytes, const tandem_outputs* out,
                          void* stream, tandem_handle** out_handle) {
  if (!out_handle) return fail(nullptr, TANDEM_E_ARG, "tandem_init: out_handle is NULL");
  *out_handle = nullptr;
  if (!senior || (junior && !sw) || !smp || !cap || !out)
    return fail(nullptr, TANDEM_E_ARG, "tandem_init: NULL argument");
  tandem_status s;
  const int nm = junior ? 2 : 1;
  if ((s = check_cfg(&senior->cfg, "senior", nullptr)) != TANDEM_OK) return s;
  if (junior && (s = check_cfg(&junior->cfg, "junior", nullptr)) != TANDEM_OK) return s;
  if (junior && senior->cfg.vocab != junior->cfg.vocab)
    return fail(nullptr, TANDEM_E_SHAPE, "senior and junior must share one vocabulary");
  if ((s = check_cap(cap, nullptr)) != TANDEM_OK) return s;
  const tandem_model* md[2] = {senior, junior};
  for (int i = 0; i < nm; ++i) {
    const tandem_model* m = md[i];
    if (!m->embed || !m->layers || !m->final_norm || !m->lm_head)
      return fail(nullptr, TANDEM_E_ARG, "tandem_init: a model weight pointer is NULL");
    auto misaligned = [](const void* p) { return ((uintptr_t)p & 15u) != 0; };
    if (misaligned(m->embed) || misaligned(m->final_norm) || misaligned(m->lm_head))
      return fail(nullptr, TANDEM_E_ARG, "tandem_init: weights must be 16-byte aligned");
    for (int l = 0; l < m->cfg.n_layers; ++l) {
      const void* const* p = m->layers + 8 * l;
      if (!p[0] || !p[1] || !p[4] || !p[5] || !p[6] || !p[7] || (m->cfg.qk_norm && (!p[2] || !p[3])))
        return fail(nullptr, TANDEM_E_ARG, "tandem_init: a layer weight pointer is NULL");
      for (int k = 0; k < 8; ++k)
        if (p[k] && misaligned(p[k])) return fail(nullptr, TANDEM_E_ARG, "tandem_init: weights must be 16-byte aligned");
    }
  }
  // The senior alone: it emits every token (SWITCH with p = 0, senior first);
  // the caller's switch settings, if any, do not apply.
  const tandem_switch_cfg solo_sw{TANDEM_SWITCH, 0.0, -1, nullptr, TANDEM_SENIOR};
  if (!junior) sw = &solo_sw;
  if (sw->mode < TANDEM_REDRAW || sw->mode > TANDEM_ALTERNATE)
    return fail(nullptr, TANDEM_E_ARG, "switch mode must be REDRAW, SWITCH or ALTERNATE");
  if (!(sw->p >= 0.0 && sw->p <= 1.0)) return fail(nullptr, TANDEM_E_ARG, "switch p must lie in [0, 1]");
  if (sw->first_owner < TANDEM_JUNIOR || sw->first_owner > TANDEM_DRAW)
    return fail(nullptr, TANDEM_E_ARG, "first_owner must be JUNIOR, SENIOR or DRAW");
  if (!(smp->temperature > 0.f) || !std::isfinite(smp->temperature))
    return fail(nullptr, TANDEM_E_ARG, "temperature must be finite and > 0");
  if (smp->eos_id >= senior->cfg.vocab) return fail(nullptr, TANDEM_E_ARG, "eos_id must be < vocab");
  if (smp->max_new_tokens < 1) return fail(nullptr, TANDEM_E_ARG, "max_new_tokens must be >= 1");
  if (smp->max_new_tokens > cap->max_ctx)
    return fail(nullptr, TANDEM_E_CAPACITY, "max_new_tokens exceeds max_ctx");
  if (!out->tokens || !out->owner || !out->senior_logprob || !out->length)
    return fail(nullptr, TANDEM_E_ARG, "tandem_init: an output arena is NULL");
  if (!kv_arena || !scratch) return fail(nullptr, TANDEM_E_ARG, "tandem_init: kv_arena or scratch is NULL");
  if (((uintptr_t)kv_arena % kAlign) || ((uintptr_t)scratch % kAlign))
    return fail(nullptr, TANDEM_E_ARG, "kv_arena and scratch must be 256-byte aligned");
  Plan P = make_plan(&senior->cfg, junior ? &junior->cfg : nullptr, cap);
  if (kv_bytes < P.kv_bytes || scratch_bytes < P.scratch_bytes)
    return fail(nullptr, TANDEM_E_CAPACITY, "kv_arena or scratch smaller than tandem_workspace_size");

  tandem_handle* h = new tandem_handle();
  h->plan = P;
  h->nm = nm;
  h->sw = *sw;
  h->smp = *smp;
  h->cap = *cap;
  h->out = *out;
  h->stream = (hipStream_t)stream;
  const double thr = std::floor(sw->p * 4294967296.0);
  h->thr = thr >= 4294967296.0 ? (1ull << 32) : (unsigned long long)thr;
  h->key0 = (uint32_t)(smp->seed & 0xFFFFFFFFull);
  h->key1 = (uint32_t)(smp->seed >> 32);
  char* kv = (char*)kv_arena;
  char* sc = (char*)scratch;
  size_t kv_off = 0;
  for (int i = 0; i < nm; ++i) {
    Model& m = h->m[i];
    const tandem_model* src = md[i];
    m.cfg = src->cfg;
    m.p = P.m[i];
    m.embed = src->embed;
    m.final_norm = (const float*)src->final_norm;
    m.lm_head = src->lm_head;
    m.layers.resize(m.cfg.n_layers);
    for (int l = 0; l < m.cfg.n_layers; ++l) {
      const void* const* p = src->layers + 8 * l;
      m.layers[l] = Layer{(const float*)p[0], p[1], (const float*)p[2], (const float*)p[3],
                          p[4], (const float*)p[5], p[6], p[7], nullptr, nullptr, nullptr, nullptr};
    }
    m.slot_stride = (long)m.cfg.n_kv_heads * P.ctx_stride * m.cfg.head_dim;
    m.layer_stride = (long)cap->max_seqs * m.slot_stride;
    m.kc = kv + kv_off;
    m.vc = kv + kv_off + m.p.kv_half;
    kv_off += 2 * m.p.kv_half;
    m.h = (float*)(sc + m.p.off_h);
    m.xa = sc + m.p.off_xa;
    m.xf = sc + m.p.off_xf;
    m.q = (float*)(sc + m.p.off_q);
    m.ws = (float*)(sc + m.p.off_ws);
    m.logits = (float*)(sc + m.p.off_logits);
    m.rope = (float2*)(sc + m.p.off_rope);
    m.p_lm = nullptr;
  }
  const size_t S = (size_t)cap->max_seqs;
  int32_t* stt = (int32_t*)(sc + P.off_state);
  h->owner = stt; h->c = stt + S; h->t = stt + 2 * S; h->pos = stt + 3 * S; h->pending = stt + 4 * S;
  h->done = stt + 5 * S;
  h->seq_slot = (int32_t*)(sc + P.off_seq_slot);
  int32_t* rows = (int32_t*)(sc + P.off_rows);
  const size_t PT = (size_t)cap->max_prefill_tokens;
  h->row_slot = rows; h->row_pos = rows + PT; h->row_tok = rows + 2 * PT;
  h->grp_row0 = rows + 3 * PT; h->grp_n = rows + 4 * PT;
  int32_t* pr = (int32_t*)(sc + P.off_prompt);
  h->p_end = pr; h->p_len = pr + S; h->p_rbase = pr + 2 * S; h->p_gbase = pr + 3 * S;
  h->d_err = (int32_t*)(sc + P.off_err);
  h->partials = (float*)(sc + P.off_partials);
  h->d_count = (int32_t*)(sc + P.off_count);
  h->act = (int32_t*)(sc + P.off_act);
  int32_t* drows = (int32_t*)(sc + P.off_drows);
  h->drow_tok = drows; h->drow_slot = drows + S; h->drow_pos = drows + 2 * S; h->drow_done = drows + 3 * S;
  h->score_part = (float*)(sc + P.off_score);
  if (P.fused) {
    h->noise = (float*)(sc + P.off_noise);
    h->part_sen = (float*)(sc + P.off_part_sen);
    h->part_jun = nm == 2 ? (float*)(sc + P.off_part_jun) : h->part_sen;
  }
  int32_t* pfx = (int32_t*)(sc + P.off_pfx);
  h->row_lo = pfx; h->pfx_slot = pfx + S;

  // --- HIP work from here on
  auto bail = [&](hipError_t e, const char* what) {
    std::string msg = std::string("HIP error in tandem_init (") + what + "): " + hipGetErrorString(e);
    if (h->h_sync) (void)hipHostFree(h->h_sync);
    if (h->h_stage) (void)hipHostFree(h->h_stage);
    if (h->ev_stage) (void)hipEventDestroy(h->ev_stage);
    for (int i = 0; i < 2; ++i)
      for (hipEvent_t ev : h->ev_att[i]) (void)hipEventDestroy(ev);
    if (h->ev_fork) (void)hipEventDestroy(h->ev_fork);
    if (h->ev_join) (void)hipEventDestroy(h->ev_join);
    if (h->ev_noise) (void)hipEventDestroy(h->ev_noise);
    if (h->side) (void)hipStreamDestroy(h->side);
    if (h->gstream) (void)hipStreamDestroy(h->gstream);
    delete h;
    return fail(nullptr, TANDEM_E_HIP, msg);
  };
  hipError_t e = hipHostMalloc((void**)&h->h_sync, 8, hipHostMallocDefault);
  if (e != hipSuccess) { h->h_sync = nullptr; return bail(e, "hipHostMalloc"); }
  e = hipHostMalloc((void**)&h->h_stage, 4 * S * 4, hipHostMallocDefault);
  if (e != hipSuccess) { h->h_stage = nullptr; return bail(e, "hipHostMalloc"); }
  e = hipEventCreateWithFlags(&h->ev_stage, hipEventDisableTiming);
  if (e != hipSuccess) { h->ev_stage = nullptr; return bail(e, "staging event"); }
  {
    int dev = 0, ncu = 0;
    e = hipGetDevice(&dev);
    if (e != hipSuccess) return bail(e, "hipGetDevice");
    e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return bail(e, "compute unit count");
    if (ncu > 0) h->n_cu = ncu;
  }
  e = hipStreamCreateWithFlags(&h->side, hipStreamNonBlocking);
  if (e != hipSuccess) { h->side = nullptr; return bail(e, "side stream"); }
  e = hipEventCreateWithFlags(&h->ev_fork, hipEventDisableTiming);
  if (e != hipSuccess) { h->ev_fork = nullptr; return bail(e, "fork event"); }
  e = hipEventCreateWithFlags(&h->ev_join, hipEventDisableTiming);
  if (e != hipSuccess) { h->ev_join = nullptr; return bail(e, "join event"); }
  e = hipEventCreateWithFlags(&h->ev_noise, hipEventDisableTiming);
  if (e != hipSuccess) { h->ev_noise = nullptr; return bail(e, "noise event"); }
  h->fused = P.fused && h->n_cu <= kSampleParts;
  e = hipStreamCreateWithFlags(&h->gstream, hipStreamNonBlocking);
  if (e != hipSuccess) { h->gstream = nullptr; return bail(e, "graph stream"); }
  for (int i = 0; i < nm; ++i)
    for (int l = 0; l < h->m[i].cfg.n_layers; ++l) {
      hipEvent_t ev;
      e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
      if (e != hipSuccess) return bail(e, "attention event");
      h->ev_att[i].push_back(ev);
    }
  for (int i = 0; i < nm; ++i) {
    e = launch_rope_table(h->m[i].cfg.rope_theta, h->m[i].cfg.head_dim, P.ctx_stride, h->m[i].rope, h->stream);
    if (e != hipSuccess) return bail(e, "rope table");
  }
  // MFMA-ordered copies of the projection and LM-head weights (read by the
  // streaming decode GEMM; the caller's row-major weights stay in use for
  // prefill-sized products)
  for (int i = 0; i < nm; ++i) {
    Model& m = h->m[i];
    char* dst = sc + m.p.off_packed;
    const auto shapes = packed_shapes(&m.cfg);
    size_t k = 0;
    const tandem_model_cfg& mc = m.cfg;
    m.ffn16 = packs(&mc, 2 * mc.ffn_dim, mc.d_model) && packs(&mc, mc.d_model, mc.ffn_dim);
    m.lm16 = packs(&mc, mc.vocab, mc.d_model);
    auto pack = [&](const void* src, int N, int K, int pair_rows, bool to_f16, const void** out) -> hipError_t {
      const auto& nk = shapes[k++];
      if (nk.first != N || nk.second != K) return hipErrorInvalidValue;
      *out = nullptr;
      if (!packs(&m.cfg, N, K)) return hipSuccess;
      hipError_t r = launch_pack_weights(src, N, K, pair_rows, to_f16, dst, h->stream);
      *out = dst;
      dst += align_up(packed_weight_bytes(N, K), kAlign);
      return r;
    };
    const tandem_model_cfg& c = m.cfg;
    for (int l = 0; l < c.n_layers && e == hipSuccess; ++l) {
      Layer& L = m.layers[l];
      if (e == hipSuccess) e = pack(L.w_qkv, m.p.qkv_dim, c.d_model, 0, false, &L.p_qkv);
      if (e == hipSuccess) e = pack(L.w_o, c.d_model, m.p.att_dim, 0, false, &L.p_o);
      if (e == hipSuccess) e = pack(L.w_gate_up, 2 * c.ffn_dim, c.d_model, c.ffn_dim, m.ffn16, &L.p_gate_up);
      if (e == hipSuccess) e = pack(L.w_down, c.d_model, c.ffn_dim, 0, m.ffn16, &L.p_down);
    }
    if (e == hipSuccess) e = pack(m.lm_head, c.vocab, c.d_model, 0, m.lm16, &m.p_lm);
    if (e != hipSuccess) return bail(e, "weight packing");
  }
  e = launch_iota(h->seq_slot, (int)S, h->stream);       // slots follow sequence ids
  if (e != hipSuccess) return bail(e, "seq slots");
  e = hipMemsetAsync(stt, 0, 6 * S * 4, h->stream);
  if (e == hipSuccess) e = hipMemsetAsync(h->d_err, 0, 4, h->stream);
  if (e != hipSuccess) return bail(e, "state");
  *out_handle = h;
  return TANDEM_OK;
}

tandem_status tandem_prefill(tandem_handle* h, const int32_t* prompt_tokens, const int32_t* prompt_offsets,
                             int32_t n_prompts, int32_t G) {
  if (!h) return fail(nullptr, TANDEM_E_ARG, "handle is NULL");
  if (h->poisoned) return fail(&h->err, TANDEM_E_STATE, "handle is poisoned by an earlier HIP error");
  if (!prompt_tokens || !prompt_offsets) return fail(&h->err, TANDEM_E_ARG, "prefill: NULL prompts");
  if (n_prompts < 1 || G < 1) return fail(&h->err, TANDEM_E_ARG, "prefill: n_prompts and G must be >= 1");
  if ((long)n_prompts * G > h->cap.max_seqs)
    return fail(&h->err, TANDEM_E_CAPACITY, "prefill: n_prompts * G exceeds max_seqs");
  if (prompt_offsets[0] != 0) return fail(&h->err, TANDEM_E_ARG, "prefill: prompt_offsets[0] must be 0");
  for (int j = 0; j < n_prompts; ++j) {
    const int P = prompt_offsets[j + 1] - prompt_offsets[j];
    if (P < 1) return fail(&h->err, TANDEM_E_ARG, "prefill: every prompt needs at least one token");
    if ((long)P - 1 + h->smp.max_new_tokens > h->cap.max_ctx)
      return fail(&h->err, TANDEM_E_CAPACITY, "prefill: prompt length - 1 + max_new_tokens exceeds max_ctx");
    if (P - 1 > h->cap.max_prefill_tokens)
      return fail(&h->err, TANDEM_E_CAPACITY, "prefill: a prompt is longer than max_prefill_tokens + 1");
  }
  hipStream_t st = h->stream;
  h->prefilled = false;
  drop_graphs(h);      // a new batch: the step graph is captured again on demand
  const int n_seq = n_prompts * G;
  // the G sequences of a prompt share its prefix in decode attention when
  // both models' attention kernels can (otherwise every slot gets a copy)
  bool share = G > 1;
  for (int i = 0; i < h->nm; ++i) {
    const tandem_model_cfg& c = h->m[i].cfg;
    share = share && attention_shares_prefix(c.weight_dtype == TANDEM_BF16 ? DT_BF16 : DT_F32, c.head_dim,
                                             c.n_q_heads / c.n_kv_heads);
  }
  h->share = share;
  h->G = G;
  // per-prompt table (exclusive end, length, first row and first 16-row group
  // within its chunk of whole prompts whose rows fit max_prefill_tokens),
  // uploaded once from pinned staging; the staging is refilled only after the
  // previous prefill's upload has left it
  std::vector<std::pair<int, int>> chunks;           // [j0, j1) per chunk
  HIPCHK(hipEventSynchronize(h->ev_stage));
  {
    int32_t* t = h->h_stage;
    int j0 = 0, nr = 0, ng = 0;
    for (int j = 0; j < n_prompts; ++j) {
      const int rows = prompt_offsets[j + 1] - prompt_offsets[j] - 1;
      if (nr + rows > h->cap.max_prefill_tokens) {
        chunks.push_back({j0, j});
        j0 = j;
        nr = ng = 0;
      }
      t[j] = prompt_offsets[j + 1];
      t[n_prompts + j] = rows + 1;
      t[2 * n_prompts + j] = nr;
      t[3 * n_prompts + j] = ng;
      nr += rows;
      ng += (rows + 15) / 16;
    }
    chunks.push_back({j0, n_prompts});
  }
  HIPCHK(hipMemsetAsync(h->d_err, 0, 4, st));
  HIPCHK(hipMemcpyAsync(h->p_end, h->h_stage, (size_t)n_prompts * 4, hipMemcpyHostToDevice, st));
  HIPCHK(hipMemcpyAsync(h->p_len, h->h_stage + n_prompts, (size_t)n_prompts * 4, hipMemcpyHostToDevice, st));
  HIPCHK(hipMemcpyAsync(h->p_rbase, h->h_stage + 2 * n_prompts, (size_t)n_prompts * 4, hipMemcpyHostToDevice, st));
  HIPCHK(hipMemcpyAsync(h->p_gbase, h->h_stage + 3 * n_prompts, (size_t)n_prompts * 4, hipMemcpyHostToDevice, st));
  HIPCHK(hipEventRecord(h->ev_stage, st));
  for (const auto& ch : chunks) {
    const int j0 = ch.first, j1 = ch.second;
    int nr = 0, ng = 0;
    for (int j = j0; j < j1; ++j) {
      const int rows = prompt_offsets[j + 1] - prompt_offsets[j] - 1;
      nr += rows;
      ng += (rows + 15) / 16;
    }
    if (nr == 0) continue;
    PrefillRowsArgs pa{};
    pa.j0 = j0; pa.n = j1 - j0; pa.G = G; pa.V = h->m[0].cfg.vocab;
    pa.prompt_tokens = prompt_tokens; pa.prompt_end = h->p_end; pa.prompt_len = h->p_len;
    pa.row_base = h->p_rbase; pa.grp_base = h->p_gbase;
    pa.row_slot = h->row_slot; pa.row_pos = h->row_pos; pa.row_tok = h->row_tok;
    pa.grp_row0 = h->grp_row0; pa.grp_n = h->grp_n; pa.err = h->d_err;
    TIMED(TANDEM_K_OTHER, launch_prefill_rows(pa, st));
    {
      FwdRows fr{nr, h->row_tok, h->row_slot, h->row_pos, nullptr};
      fr.grp_row0 = h->grp_row0; fr.grp_n = h->grp_n; fr.n_groups = ng;
      tandem_status s = forward_pair(h, fr, false);
      if (s != TANDEM_OK) return s;
    }
    for (int j = j0; j < j1; ++j) {
      const int P = prompt_offsets[j + 1] - prompt_offsets[j];
      if (P - 1 <= 0 || G <= 1) continue;
      const int lo = share ? (P - 1) / 16 * 16 : 0;    // shared positions stay in the first slot only
      for (int i = 0; i < h->nm; ++i) {
        Model& m = h->m[i];
        TIMED(TANDEM_K_OTHER, launch_kv_replicate(m.cfg.weight_dtype == TANDEM_BF16 ? DT_BF16 : DT_F32, m.kc, m.vc,
                                   m.cfg.n_layers, m.layer_stride, m.slot_stride, m.cfg.n_kv_heads,
                                   m.cfg.head_dim, h->plan.ctx_stride, j * G, j * G + 1, G - 1, lo, P - 1, st));
      }
    }
  }
  InitStateArgs is{};
  is.n_seq = n_seq; is.G = G; is.V = h->m[0].cfg.vocab;
  is.prompt_tokens = prompt_tokens; is.prompt_end = h->p_end; is.prompt_len = h->p_len;
  is.key0 = h->key0; is.key1 = h->key1; is.thr = h->thr; is.first_owner = h->sw.first_owner;
  is.owner = h->owner; is.c = h->c; is.t = h->t; is.pos = h->pos; is.pending = h->pending; is.done = h->done;
  is.out_len = h->out.length; is.err = h->d_err;
  HIPCHK(launch_init_state(is, st));
  HIPCHK(hipMemcpyAsync(h->act, h->seq_slot, (size_t)n_seq * 4, hipMemcpyDeviceToDevice, st));   // identity
  h->n_seq = n_seq;
  h->R_launch = n_seq;
  CALL(prefix_tables(h));
  h->steps_since_compact = 0;
  h->prefilled = true;
  h->stepped = false;
  return TANDEM_OK;
}

tandem_status tandem_step(tandem_handle* h, int32_t* n_active) { return step_impl(h, nullptr, nullptr, n_active); }

tandem_status tandem_step_forced(tandem_handle* h, const int32_t* forced, const tandem_debug* dbg,
                                 int32_t* n_active) {
  if (h && !forced) return fail(&h->err, TANDEM_E_ARG, "tandem_step_forced: forced is NULL");
  return step_impl(h, forced, dbg, n_active);
}

tandem_status tandem_score_step(tandem_handle* h, float* scores) {
  if (!h) return fail(nullptr, TANDEM_E_ARG, "handle is NULL");
  if (h->poisoned) return fail(&h->err, TANDEM_E_STATE, "handle is poisoned by an earlier HIP error");
  if (!scores) return fail(&h->err, TANDEM_E_ARG, "tandem_score_step: scores is NULL");
  if (!h->prefilled || !h->stepped)
    return fail(&h->err, TANDEM_E_STATE, "tandem_score_step before a step of the current batch");
  if (h->nm != 2) return fail(&h->err, TANDEM_E_STATE, "tandem_score_step needs a junior (the handle has none)");
  // the step's rows: its act order, launched row count, done-at-start flags and
  // LM-head input rows are all still in place (compaction runs at the start of
  // a step); a step that sampled inside the LM heads stored no logits, so the
  // two heads run again here
  if (h->last_fused) {
    hipStream_t st = h->stream;
    FwdRows fr{h->R_launch, h->drow_tok, h->drow_slot, h->drow_pos, h->drow_done};
    for (int i = 0; i < 2; ++i) CALL(forward_head(h, i, fr, false, st));
    h->last_fused = false;              // the step's logits are stored now
  }
  ScoreArgs a{};
  a.z_sen = h->m[0].logits; a.z_jun = h->m[1].logits; a.R = h->R_launch; a.V = h->m[0].cfg.vocab;
  a.act = h->act; a.row_done = h->drow_done; a.tok = h->pending;
  a.lse = h->score_part;
  a.sums = a.lse + (size_t)h->cap.max_seqs * h->plan.n_chunks * 4;
  a.chunk = kVocabChunk; a.n_chunks = h->plan.n_chunks;
  a.out = scores;
  HIPCHK(launch_score(a, h->stream));
  return TANDEM_OK;
}

tandem_status tandem_get_state(tandem_handle* h, int32_t* owner, int32_t* c, int32_t* t, int32_t* pos,
                               int32_t* done) {
  if (!h) return fail(nullptr, TANDEM_E_ARG, "handle is NULL");
  if (h->poisoned) return fail(&h->err, TANDEM_E_STATE, "handle is poisoned by an earlier HIP error");
  if (!h->prefilled) return fail(&h->err, TANDEM_E_STATE, "tandem_get_state before tandem_prefill");
  const size_t n = (size_t)h->n_seq * 4;
  CALL(sync_read(h, nullptr));
  if (owner) HIPCHK(hipMemcpy(owner, h->owner, n, hipMemcpyDeviceToHost));
  if (c) HIPCHK(hipMemcpy(c, h->c, n, hipMemcpyDeviceToHost));
  if (t) HIPCHK(hipMemcpy(t, h->t, n, hipMemcpyDeviceToHost));
  if (pos) HIPCHK(hipMemcpy(pos, h->pos, n, hipMemcpyDeviceToHost));
  if (done) HIPCHK(hipMemcpy(done, h->done, n, hipMemcpyDeviceToHost));
  return TANDEM_OK;
}

tandem_status tandem_timing_enable(tandem_handle* h, int32_t class_mask) {
  if (!h) return fail(nullptr, TANDEM_E_ARG, "handle is NULL");
  if (h->poisoned) return fail(&h->err, TANDEM_E_STATE, "handle is poisoned by an earlier HIP error");
  HIPCHK(hipStreamSynchronize(h->stream));
  h->timing = class_mask & (((1 << TANDEM_K_CLASSES) - 1) | TANDEM_TIMING_SERIAL | TANDEM_TIMING_EAGER |
                            TANDEM_TIMING_SEPARATE_SAMPLE);
  h->ev_used = 0;
  h->ev_marks.clear();
  for (int k = 0; k < TANDEM_K_CLASSES; ++k) {
    h->acc_ms[k] = 0.0;
    h->acc_n[k] = 0;
  }
  return TANDEM_OK;
}

tandem_status tandem_timing_read(tandem_handle* h, int32_t kernel_class, double* total_ms, int64_t* launches) {
  if (!h) return fail(nullptr, TANDEM_E_ARG, "handle is NULL");
  if (kernel_class < 0 || kernel_class >= TANDEM_K_CLASSES || !total_ms || !launches)
    return fail(&h->err, TANDEM_E_ARG, "tandem_timing_read: bad kernel class or NULL output");
  if (h->poisoned) return fail(&h->err, TANDEM_E_STATE, "handle is poisoned by an earlier HIP error");
  HIPCHK(harvest_all(h));
  *total_ms = h->acc_ms[kernel_class];
  *launches = h->acc_n[kernel_class];
  return TANDEM_OK;
}

void tandem_destroy(tandem_handle* h) {
  if (!h) return;
  (void)hipStreamSynchronize(h->stream);
  if (h->side) (void)hipStreamSynchronize(h->side);
  if (h->gstream) (void)hipStreamSynchronize(h->gstream);
  drop_graphs(h);
  for (hipEvent_t e : h->ev_pool) (void)hipEventDestroy(e);
  for (int i = 0; i < 2; ++i)
    for (hipEvent_t e : h->ev_att[i]) (void)hipEventDestroy(e);
  if (h->ev_fork) (void)hipEventDestroy(h->ev_fork);
  if (h->ev_join) (void)hipEventDestroy(h->ev_join);
  if (h->ev_noise) (void)hipEventDestroy(h->ev_noise);
  if (h->side) (void)hipStreamDestroy(h->side);
  if (h->gstream) (void)hipStreamDestroy(h->gstream);
  if (h->h_sync) (void)hipHostFree(h->h_sync);
  if (h->h_stage) (void)hipHostFree(h->h_stage);
  if (h->ev_stage) (void)hipEventDestroy(h->ev_stage);
  delete h;
}


tandem_status tandem_grpo_workspace_size(const tandem_grpo_cfg* cfg, size_t* bytes) {
  if (!bytes) return fail(nullptr, TANDEM_E_ARG, "tandem_grpo_workspace_size: bytes is NULL");
  GrpoArgs a{};
  return grpo_check(cfg, bytes, &a);
}

tandem_status tandem_grpo_loss(const tandem_grpo_cfg* cfg, const float* rewards, const uint8_t* owner,
                               const int32_t* length, const float* logp_old, const float* logp_new,
                               float* advantages, float* grad, float* loss, int32_t* n_masked,
                               void* workspace, size_t workspace_bytes, void* stream) {
  GrpoArgs a{};
  size_t need = 0;
  const tandem_status st = grpo_check(cfg, &need, &a);
  if (st != TANDEM_OK) return st;
  if (!rewards || !owner || !length || !logp_old || !advantages || !loss || !n_masked || !workspace)
    return fail(nullptr, TANDEM_E_ARG, "tandem_grpo_loss: a required pointer is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0)
    return fail(nullptr, TANDEM_E_ARG, "tandem_grpo_loss: workspace must be 256-byte aligned");
  if (workspace_bytes < need)
    return fail(nullptr, TANDEM_E_ARG, "tandem_grpo_loss: workspace is smaller than tandem_grpo_workspace_size");
  a.rewards = rewards; a.owner = owner; a.length = length; a.logp_old = logp_old; a.logp_new = logp_new;
  a.adv = advantages; a.grad = grad; a.loss = loss; a.n_masked = n_masked;
  a.cnt = static_cast<int32_t*>(workspace);
  a.part = reinterpret_cast<float*>(static_cast<char*>(workspace) + ((size_t)a.S * 4 + 255) / 256 * 256);
  a.ticket = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + need - 256);
  const hipError_t e = launch_grpo(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess)
    return fail(nullptr, TANDEM_E_HIP, std::string("tandem_grpo_loss: ") + hipGetErrorString(e));
  return TANDEM_OK;
}

tandem_status tandem_grpo_loss_noalloc(const tandem_grpo_cfg* cfg, const float* rewards, const uint8_t* owner,
                                       const int32_t* length, const float* logp_old, const float* logp_new,
                                       float* advantages, float* grad, float* loss, int32_t* n_masked,
                                       void* stream) {
  GrpoArgs a{};
  size_t need = 0;
  const tandem_status st = grpo_check(cfg, &need, &a);
  if (st != TANDEM_OK) return st;
  if (!rewards || !owner || !length || !logp_old || !advantages || !loss || !n_masked)
    return fail(nullptr, TANDEM_E_ARG, "tandem_grpo_loss_noalloc: a required pointer is NULL");
  if (need > kGrpoStaticBytes) {
    char b[200];
    snprintf(b, sizeof b,
             "tandem_grpo_loss_noalloc: this batch needs %zu bytes of workspace, the library's device array holds "
             "%zu; use tandem_grpo_loss with a workspace",
             need, kGrpoStaticBytes);
    return fail(nullptr, TANDEM_E_CAPACITY, b);
  }
  void* ws = nullptr;
  hipError_t e = grpo_static_workspace(&ws);
  if (e != hipSuccess)
    return fail(nullptr, TANDEM_E_HIP, std::string("tandem_grpo_loss_noalloc: workspace address: ") +
                                           hipGetErrorString(e));
  a.rewards = rewards; a.owner = owner; a.length = length; a.logp_old = logp_old; a.logp_new = logp_new;
  a.adv = advantages; a.grad = grad; a.loss = loss; a.n_masked = n_masked;
  a.cnt = static_cast<int32_t*>(ws);
  a.part = reinterpret_cast<float*>(static_cast<char*>(ws) + ((size_t)a.S * 4 + 255) / 256 * 256);
  a.ticket = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + need - 256);
  e = launch_grpo(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess)
    return fail(nullptr, TANDEM_E_HIP, std::string("tandem_grpo_loss_noalloc: ") + hipGetErrorString(e));
  return TANDEM_OK;
}
}  // extern "C"
