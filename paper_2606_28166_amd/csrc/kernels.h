// Host-side launchers of the gfx950 kernels (internal to libtandem).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tandem {

enum DType { DT_BF16 = 0, DT_F32 = 1 };
enum Epi { EPI_PARTIAL = 0, EPI_STORE = 1, EPI_SWIGLU = 2, EPI_SAMPLE = 3 };

// The sampling epilogue of a decode LM head on the streaming GEMM
// (EPI_SAMPLE): instead of storing the logits z[r][v] it folds each
// workgroup's vocabulary entries into per-row partials, part[r][wg][5] =
// (max, sum of e^(s - max)) of the scores s = (z + b 1[v = eos]) / T (senior
// head only), and the top two of s + noise[r][v] with the best index, for
// the rows this model owns (owner[act[r]] == model).  wg < the launch grid.
struct SampleEpiArgs {
  const float* noise;          // [R][V] Gumbel noise of this step
  const int32_t* act;          // [R] sequence of each row
  const int32_t* owner;        // by sequence: 1 = senior
  const int32_t* done;         // by sequence
  int model;                   // 1: senior head (log-sum-exp of every row), 0: junior head
  float temp; int eos_id; float eos_bias;
  float* part;                 // [R][n_part][5]
  int n_part;                  // partials per row (>= the launch grid)
};

// C[M x N] = A[M x K] . W[N x K]^T, A fp32, W in the weight dtype.
//   EPI_PARTIAL: split-K partial sums to out + split * split_stride, row stride ldo
//   EPI_STORE:   out[m * ldo + n], splits must be 1
//   EPI_SWIGLU:  W has 2N rows (gate rows then up rows); out[m * ldo + j] =
//                silu(gate_j) * up_j for j < N
// splits is the number of K slices (>= 1); *splits_used returns the number
// actually used (may be lower when K is short).
struct GemmArgs {
  int dt;                 // weight dtype
  const void* A;          // activations [M][K] (split for bf16 weights, else fp32; fp16 when a16)
  const void* W;          // weights [rows][K]
  const void* Wp;         // the packed copy of W (bf16 models, M > 64), or NULL
  bool a16;               // fp16 activations against an fp16 packed copy (Wp required)
  int M, N, K;
  int epi;
  float* out;             // EPI_SWIGLU: activation rows of width ldo (split for bf16)
  int ldo;
  long split_stride;
  int splits;
};
hipError_t launch_gemm(const GemmArgs& a, int* splits_used, hipStream_t st);

// The K dimension granule of the MFMA path; other K use the VALU path.
constexpr int kGemmBK = 64;

// Decode projections over packed weights (k_stream.hip), M <= kStreamMaxRows.
// Packed layout of a [N][K] bf16 matrix: fragments of 32 rows x 16 k, 1 KB
// each, ordered [row block][k step]; lane l of fragment (nb, ks) holds
// W[32 nb + l % 32][16 ks + 8 (l / 32) .. +7] (rows >= N are zero).
constexpr int kStreamMaxRows = 128;
constexpr int kStreamStages = 4;   // prefetch ring depth (register sets, LDS stages); K % 256 == 0, chunks per K slice % 4 == 0
constexpr int kSplitMaxStream = 16;  // K slices at most (the consumers sum up to 16 partials)
size_t packed_weight_bytes(int N, int K);
bool stream_gemm_ok(int M, int N, int K);
// pair_rows F > 0: W is a [2F][K] gate/up matrix, packed pair-interleaved (block b =
// gate rows 16 b .. +15, then up rows F + 16 b .. +15) for the SwiGLU epilogue.
// to_f16: the copy holds fp16 values (for fp16 activations; bf16 -> fp16 is
// exact down to 2^-17 in magnitude, smaller weights round to the fp16
// subnormal grid, 2^-24).
hipError_t launch_pack_weights(const void* W, int N, int K, int pair_rows, bool to_f16, void* out, hipStream_t st);
struct StreamPlan {
  int nbw;                // 32-row weight blocks per wave (1)
  int S;                  // K slices (split-K partial tiles when > 1)
  int cps;                // 64-wide k chunks per slice
  int n_groups;           // weight-row groups of 128 * nbw rows
  int grid;               // workgroups (<= items)
};
// Chooses the blocking for an M x N x K decode projection on n_cu compute
// units.  kPlanStore: one K slice (plain output); kPlanPartial: split-K
// partials (S * M * N <= ws_floats); kPlanSwiglu: S = 1 is the fused SwiGLU
// epilogue, S > 1 partials plus a separate SwiGLU pass.
enum { kPlanStore = 0, kPlanPartial = 1, kPlanSwiglu = 2 };
StreamPlan plan_stream_gemm(int M, int N, int K, int n_cu, size_t ws_floats, int mode);
struct GemmStreamArgs {
  const void* A;          // activations: split [M][2K] (bf16 hi/lo pieces), or fp16 [M][K] when a16
  const void* Wp;         // packed weights (pair-interleaved for EPI_SWIGLU), fp16 values when a16
  int M, N, K;
  bool a16;               // fp16 activations and weights
  int epi;                // EPI_PARTIAL / EPI_STORE: out + s * split_stride + m * ldo + n;
                          // EPI_SWIGLU (S = 1): rows of ldo = N / 2 outputs, fp16 when
                          // a16, split format otherwise
  float* out;
  int ldo;
  long split_stride;
  int nbw, S, cps, n_groups, grid;
  SampleEpiArgs smp;      // EPI_SAMPLE (a16, S = 1)
};
hipError_t launch_gemm_stream(const GemmStreamArgs& a, hipStream_t st);

// Activations x feeding a GEMM are in split format for bf16 models (see
// common.h) and plain fp32 for fp32 models; both take 4 bytes per value.
// The streaming decode GEMMs of the FFN and the LM head take fp16 rows
// instead (f16_out below: [R][d] of 2-byte values).

// h[r] = E[tok[r]], x[r] = rmsnorm(h[r]) * gain.
hipError_t launch_embed_norm(int dt, const int32_t* tok, const void* E, int d, const float* gain,
                             float eps, float* h, void* x, int R, hipStream_t st);

// h[r] += sum_s ws[s][r] (fixed order), then x[r] = rmsnorm(h[r]) * gain.
// SwiGLU of split-K gate/up partials: ws[s][m][0 .. ffn) are gate sums,
// ws[s][m][ffn .. 2 ffn) the matching up sums; out[m] = silu(gate) * up in
// split format (row stride 2 * ffn bf16), or fp16 (row stride ffn) when
// f16_out.  ffn % 8 == 0.
// interleaved: the partial columns follow the pair-interleaved packing (gate
// j at 32 (j / 16) + j % 16, up j 16 columns later).
hipError_t launch_swiglu_finish(const float* ws, int S, long ws_stride, int M, int ffn, bool interleaved, bool f16_out,
                                void* out, hipStream_t st);

hipError_t launch_resid_norm(int dt, const float* ws, int S, long ws_stride, float* h,
                             const float* gain, float eps, void* x, int R, int d, bool f16_out, hipStream_t st);

struct CacheGeom {
  void* k;                // layer base of the K cache  [slot][kvh][tiled plane of ctx_stride x hd]
  void* v;                // layer base of the V cache  [slot][kvh][tiled plane of ctx_stride x hd]
  int ctx_stride;
  long slot_stride;       // elements between slots (= n_kv * ctx_stride * hd)
};

// Sum the QKV split-K partials, per-head RMSNorm of q and k (optional), RoPE,
// write q (fp32) and append k, v to the cache (weight dtype, rounded to
// nearest even for bf16) at (slot, pos).
struct QkvPostArgs {
  int dt;
  const float* ws; int S; long ws_stride;
  int R, nq, nkv, hd;
  const float* q_norm; const float* k_norm; float eps;
  const float2* rope;     // [ctx_stride][hd/2] (cos, sin)
  const int32_t* row_slot; const int32_t* row_pos; const int32_t* row_done;
  float* q_out;           // [R][nq][hd]
  CacheGeom cache;
};
hipError_t launch_qkv_post(const QkvPostArgs& a, hipStream_t st);

// Decode/prefill attention of every row's query heads over positions
// 0..row_pos[r] of its slot; out[r][h * hd + d] (an activation row of width
// nq * hd, split for bf16 models).
struct AttnArgs {
  int dt;
  const float* q; int R, nq, nkv, hd;
  CacheGeom cache;
  const int32_t* row_slot; const int32_t* row_pos; const int32_t* row_done;
  void* out;
  // prompt rows (row_done NULL): n_groups groups of at most 16 consecutive
  // rows of one prompt, rows grp_row0[g] .. + grp_n[g] - 1 in increasing
  // position order; NULL: one workgroup per row
  const int32_t* grp_row0; const int32_t* grp_n; int n_groups;
  // Decode rows whose prompt prefix is shared (row_lo != NULL; needs
  // row_done): row r attends positions [0, row_lo[r]) in slot pfx_slot[r]
  // and [row_lo[r], row_pos[r]] in its own slot; row_lo is a multiple of 16
  // (0: the whole context in the row's own slot).
  const int32_t* row_lo; const int32_t* pfx_slot;
};
hipError_t launch_attention(const AttnArgs& a, hipStream_t st);

// rope table [n_pos][hd/2] of (cos, sin)(pos * theta^(-2i/hd)), computed in fp64.
hipError_t launch_rope_table(float theta, int hd, int n_pos, float2* out, hipStream_t st);

// Sampling.
struct SampleArgs {
  const float* z_sen;     // [R][V]
  const float* z_jun;     // [R][V]
  int R, V;
  float temp; int eos_id; float eos_bias_sen, eos_bias_jun;
  uint32_t key0, key1;
  const int32_t* owner; const int32_t* t; const int32_t* done;   // per sequence
  const int32_t* act;     // [R] sequence of each row
  float* partials;        // [R][n_chunks][5]
  int chunk;              // vocab entries per chunk
};
hipError_t launch_sample_partials(const SampleArgs& a, int n_chunks, hipStream_t st);

// Gumbel noise of this step for launched rows 0 .. R-1 that are not done:
// noise[r][v] = -log(-log u) of the token stream's Philox word for (seed,
// sequence act[r], step t, v) (the same words sample_partials draws).
// V % 4 == 0.
hipError_t launch_gumbel_noise(const int32_t* act, const int32_t* t, const int32_t* done, int R, int V,
                               uint32_t key0, uint32_t key1, float* noise, hipStream_t st);

struct FinishArgs {
  const float* z_sen; int R, V;           // logits by row
  const int32_t* act;                     // [R] sequence of each row (state and outputs by sequence)
  float temp; int eos_id; float eos_bias_sen;
  const float* partials; int n_chunks;
  const int32_t* forced;                      // [R] or NULL
  uint32_t key0, key1; unsigned long long thr; int mode; int cap_k;
  const uint32_t* bnd;                        // NULL = all boundaries
  int max_new;
  int32_t* owner; int32_t* c; int32_t* t; int32_t* pos; int32_t* pending; int32_t* done;
  int32_t* out_tok; uint8_t* out_own; float* out_lp; int32_t* out_len; int ld_out;
  int32_t* dbg_sampled; float* dbg_margin;
  int32_t* n_active;                          // device counter or NULL
  // Sampling-epilogue partials instead of the logits (part_sen != NULL):
  // the senior head's n_sen partials per row (log-sum-exp, and top two for
  // senior-owned rows), the junior head's n_jun (top two for junior-owned
  // rows); the chosen token's senior score is recomputed from the senior's
  // LM-head input rows x_sen (fp16 [R][d]) and its bf16 LM head w_lm [V][d].
  const float* part_sen; int n_sen; const float* part_jun; int n_jun;
  const uint16_t* x_sen; const uint16_t* w_lm; int d;
};
hipError_t launch_sample_finish(const FinishArgs& a, hipStream_t st);

// Dual-distribution scores of the rows of the step just taken, from both
// models' logits [R][V] (temperature 1, no bias): per sequence act[r] of a
// row not done before the step (row_done[r] == 0), with y = tok[act[r]]
// the token the step emitted, out[act[r]][0 .. 2] = (-log p_jun(y),
// sum_v min(p_sen, p_jun), KL(p_sen || p_jun)).  lse: [R][n_chunks][4],
// sums: [R][n_chunks][2] of scratch; chunk vocabulary entries per chunk.
struct ScoreArgs {
  const float* z_sen; const float* z_jun; int R, V;
  const int32_t* act; const int32_t* row_done; const int32_t* tok;
  float* lse; float* sums; int chunk, n_chunks;
  float* out;
};
hipError_t launch_score(const ScoreArgs& a, hipStream_t st);

// Senior-only GRPO loss pieces over S = n_groups * G rollouts with arenas of
// row stride T: advantages adv[S], masked counts cnt[S] (scratch), per-(row,
// chunk) partial sums part[S][n_chunks] (scratch, n_chunks = ceil(T /
// kGrpoChunk)), a completion ticket (scratch, zeroed by the first launch),
// gradient grad[S][T] (may be NULL), loss[1], n_masked[1].
// logp_new NULL means logp_new = logp_old.
constexpr int kGrpoChunk = 1024;
struct GrpoArgs {
  int S, G, T, n_chunks; float eps;
  const float* rewards; const uint8_t* owner; const int32_t* length;
  const float* logp_old; const float* logp_new;
  float* adv; int32_t* cnt; float* part; int32_t* ticket; float* grad; float* loss; int32_t* n_masked;
};
hipError_t launch_grpo(const GrpoArgs& a, hipStream_t st);
// Bytes of the device-resident workspace of the allocation-free GRPO entry
// point, and its device address on the current device (looked up once per
// device).
constexpr size_t kGrpoStaticBytes = (size_t)1 << 20;
hipError_t grpo_static_workspace(void** ptr);

// Copy positions [p0, n_pos) of slot src into slots dst0 .. dst0 + n_dst - 1
// for every layer and kv head (K and transposed V); p0 % 16 == 0.
hipError_t launch_kv_replicate(int dt, void* kc, void* vc, int n_layers, long layer_stride,
                               long slot_stride, int nkv, int hd, int ctx_stride, int src,
                               int dst0, int n_dst, int p0, int n_pos, hipStream_t st);

// Per-sequence state after prefill.  The pending token (a prompt's last
// token) is range-checked like the prompt rows (see PrefillRowsArgs).
struct InitStateArgs {
  int n_seq, G, V;
  const int32_t* prompt_tokens; const int32_t* prompt_end;   // device [n_prompts] exclusive ends
  const int32_t* prompt_len;                                 // device [n_prompts]
  uint32_t key0, key1; unsigned long long thr; int first_owner;
  int32_t* owner; int32_t* c; int32_t* t; int32_t* pos; int32_t* pending; int32_t* done;
  int32_t* out_len;
  int32_t* err;                                              // set to 1 when a token id is outside [0, V)
};

// Row tables of one prefill chunk, prompts j0 .. j0 + n - 1: prompt j's
// P_j - 1 rows start at row_base[j] (chunk-relative) with slot j G,
// positions 0 .. P_j - 2 and tokens prompt_tokens[end_j - P_j + i]; its
// groups of 16 rows start at grp_base[j].  A token id outside [0, V) is
// replaced by 0 (so every later read stays in bounds) and sets *err.
struct PrefillRowsArgs {
  int j0, n, G, V;
  const int32_t* prompt_tokens;
  const int32_t* prompt_end; const int32_t* prompt_len;      // device [n_prompts]
  const int32_t* row_base; const int32_t* grp_base;          // device [n_prompts]
  int32_t* row_slot; int32_t* row_pos; int32_t* row_tok; int32_t* grp_row0; int32_t* grp_n;
  int32_t* err;
};
hipError_t launch_prefill_rows(const PrefillRowsArgs& a, hipStream_t st);

// dst[i] = i for i < n.
hipError_t launch_iota(int32_t* dst, int n, hipStream_t st);

// Shared-prefix tables of decode rows 0 .. R-1: row r of sequence act[r]
// (prompt j = act[r] / G) reads positions [0, lo) from slot j G, lo =
// (P_j - 1) rounded down to 16.
hipError_t launch_prefix_rows(const int32_t* act, int R, int G, const int32_t* prompt_len, int32_t* row_lo,
                              int32_t* pfx_slot, hipStream_t st);
hipError_t launch_init_state(const InitStateArgs& a, hipStream_t st);

hipError_t launch_count_active(const int32_t* done, int n, int32_t* out, hipStream_t st);

// Stable partition of the sequence ids 0 .. n-1: act[0 .. n_active) = the
// unfinished ones in increasing order, then the finished ones in increasing
// order; *n_active_out = their count.  One workgroup.
hipError_t launch_compact(const int32_t* done, int n, int32_t* act, int32_t* n_active_out, hipStream_t st);

// Decode row arrays for rows 0 .. R-1 from the row -> sequence map.
struct GatherRowsArgs {
  const int32_t* act; int R;
  const int32_t* pending; const int32_t* seq_slot; const int32_t* pos; const int32_t* done;
  int32_t* row_tok; int32_t* row_slot; int32_t* row_pos; int32_t* row_done;
};
hipError_t launch_gather_rows(const GatherRowsArgs& a, hipStream_t st);

// dst[act[r]][0 .. V) = src[r][0 .. V) for rows 0 .. R-1 (debug logits by sequence).
hipError_t launch_scatter_rows(const float* src, const int32_t* act, int R, int V, float* dst, hipStream_t st);


// true when the MFMA attention kernel covers this (dtype, head_dim, group size)
bool attention_has_mfma(int dt, int hd, int gqa);
// true when decode attention can read a shared prompt prefix once per row block
bool attention_shares_prefix(int dt, int hd, int gqa);

}  // namespace tandem
