// Grouped-query attention of one new query position per row over that row's
// KV cache (decode), also used for prompt rows (each prompt token attends to
// positions 0..its own position of the prompt's cache).
//
// bf16 path (HD in {64, 128}): one workgroup per (kv head, row); its four
// waves take interleaved 16-position chunks of the tiled cache and keep
// their own online softmax, merged through LDS at the end.  The products
// run on MFMA:
//   S^T = K . Q^T   16x16x32: A = 16 cached keys x 32 dims, B = 32 dims x 16
//                   query heads of the group (heads >= G are zero);
//   O  += P . V     16x16x16: A = 16 heads x 16 positions, which is exactly
//                   the S^T accumulator layout (lane (g, c) holds positions
//                   4g .. 4g+3 of head c), B = 16 positions x 16 dims.
// The fp32 query and the fp32 softmax weights enter as bf16 high + low parts
// (two MFMAs each), so only the cache itself is bf16.  The cache is tiled in
// operand order: every load is one contiguous 1 KB piece per wave, issued
// as a non-temporal buffer load one chunk ahead of the arithmetic.  One load
// of a kv head's keys serves all G query heads of its group.
//
// fp32 path: a plain VALU kernel, one workgroup per (query head, row).
#include "common.h"
#include "kernels.h"


namespace tandem {

namespace {

typedef short s16x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void split8(const float* x, bf16x8_t& hi, bf16x8_t& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const bf16_t h0 = f2bf(x[2 * e]), h1 = f2bf(x[2 * e + 1]);
    const bf16_t l0 = f2bf(x[2 * e] - bf2f(h0)), l1 = f2bf(x[2 * e + 1] - bf2f(h1));
    h[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
    l[e] = (uint32_t)l0 | ((uint32_t)l1 << 16);
  }
  hi = __builtin_bit_cast(bf16x8_t, make_uint4(h[0], h[1], h[2], h[3]));
  lo = __builtin_bit_cast(bf16x8_t, make_uint4(l[0], l[1], l[2], l[3]));
}

// 4 fp32 -> bf16 high parts and bf16 low parts (x ~ hi + lo), as MFMA operands
__device__ __forceinline__ void split4(const float* x, s16x4_t& hi, s16x4_t& lo) {
  uint32_t h[2], l[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const bf16_t h0 = f2bf(x[2 * e]), h1 = f2bf(x[2 * e + 1]);
    const bf16_t l0 = f2bf(x[2 * e] - bf2f(h0)), l1 = f2bf(x[2 * e + 1] - bf2f(h1));
    h[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
    l[e] = (uint32_t)l0 | ((uint32_t)l1 << 16);
  }
  hi = __builtin_bit_cast(s16x4_t, make_uint2(h[0], h[1]));
  lo = __builtin_bit_cast(s16x4_t, make_uint2(l[0], l[1]));
}

// One 16-position chunk of a kv head's keys and values in MFMA operand
// layout (the cache's tiled order): k[dc] = K[pos c16][32dc + 8g .. +7];
// v[j] = V[pos 4g .. +3][32j + c16] then V[pos 4g .. +3][32j + 16 + c16].
// Half a 16-position chunk: its K or its V tile (16 positions x HD, bf16)
// in the lane order the MFMAs consume, 16 bytes per lane per 32 dims.
template <int HD>
struct Half {
  u32x4_t r[HD / 32];
};

template <int HD, bool NT = true>
__device__ __forceinline__ void load_half(Half<HD>& h, __amdgpu_buffer_rsrc_t rs, int chunk, int lane) {
  const int base = chunk * 32 * HD + lane * 16;   // bytes: 16 positions x HD x 2
#pragma unroll
  for (int j = 0; j < HD / 32; ++j) h.r[j] = NT ? buf_load16_nt(rs, base + j * 1024, 0) : buf_load16(rs, base + j * 1024, 0);
}

// Orders the loads issued so far before everything that follows and ties h
// to this point: the empty asm "modifies" every register of h and clobbers
// memory, so earlier loads cannot sink below it, later loads cannot rise
// above it, arithmetic on h cannot cross it, and the only wait the compiler
// places here is for h's own loads.
template <int HD>
__device__ __forceinline__ void pin_half(Half<HD>& h) {
#pragma unroll
  for (int j = 0; j < HD / 32; ++j) asm volatile("" : "+v"(h.r[j]) : : "memory");
}

template <int HD>
struct AttnState {
  float m_run, l_run;             // running max (log2 units) and this lane's share of the sum
  f32x4_t o[HD / 16];             // O[head 4g + i][dim 16 db + c16]
};

// ctx: this lane's query column attends positions < ctx; ctx_max: positions
// >= ctx_max hold stale cache contents.  GUARD: a column may see a chunk with
// no position it attends before any it does (several query rows per
// workgroup); its running max then stays -inf and nothing is added.
// First half of a chunk: scores of its 16 positions from the K tile, the
// online-softmax update and the rescaling of the accumulator; returns the
// probabilities as split bf16 operands of the value product.
template <int HD, bool GUARD>
__device__ __forceinline__ void attend_scores(AttnState<HD>& st, const Half<HD>& k, const bf16x8_t* qh,
                                              const bf16x8_t* ql, int p0, int ctx, float scale, int g, s16x4_t& ph,
                                              s16x4_t& pl) {
  constexpr int DC = HD / 32, DB = HD / 16;
  f32x4_t acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int dc = 0; dc < DC; ++dc) {
    const bf16x8_t kk = __builtin_bit_cast(bf16x8_t, k.r[dc]);
    acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, qh[dc], acc0, 0, 0, 0);
    acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, ql[dc], acc1, 0, 0, 0);
  }
  // lane (g, c16): scores of positions p0 + 4g + i for head c16
  const int pg = p0 + 4 * g;
  float s[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) s[i] = pg + i < ctx ? (acc0[i] + acc1[i]) * scale : -INFINITY;
  float mx = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  const float m_new = fmaxf(st.m_run, mx);
  const bool none = GUARD && m_new == -INFINITY;
  const float alpha = none ? 1.f : exp2f(st.m_run - m_new);
  float pr[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) pr[i] = none ? 0.f : exp2f(s[i] - m_new);
  st.l_run = st.l_run * alpha + ((pr[0] + pr[1]) + (pr[2] + pr[3]));
  st.m_run = m_new;
  split4(pr, ph, pl);
  // rescale the accumulator rows (heads 4g + i) only when some head's max moved
  if (__ballot(alpha != 1.f)) {
    float ai[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) ai[i] = __shfl(alpha, 4 * g + i, 64);
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) st.o[db][i] *= ai[i];
  }
}

// Second half of a chunk: the probabilities times its V tile.
template <int HD>
__device__ __forceinline__ void attend_values(AttnState<HD>& st, Half<HD>& v, s16x4_t ph, s16x4_t pl, int p0,
                                              int ctx_max, int g) {
  constexpr int DC = HD / 32, DB = HD / 16;
  const int pg = p0 + 4 * g;
  // positions at or past the context hold stale cache contents: zero them so
  // that 0 * (stale) cannot produce NaN
  if (p0 + 16 > ctx_max) {
    // keep the first nv of this lane's four positions (16 bits each)
    const int nv = min(max(ctx_max - pg, 0), 4);
    const uint64_t keep = nv == 4 ? ~0ull : (1ull << (16 * nv)) - 1ull;
    const uint32_t klo = (uint32_t)keep, khi = (uint32_t)(keep >> 32);
#pragma unroll
    for (int j = 0; j < DC; ++j) v.r[j] &= u32x4_t{klo, khi, klo, khi};
  }
  // hi parts over all dim blocks, then lo parts (independent consecutive MFMAs)
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const u32x4_t w = v.r[db >> 1];
    const s16x4_t vv = __builtin_bit_cast(s16x4_t, (db & 1) ? make_uint2(w.z, w.w) : make_uint2(w.x, w.y));
    st.o[db] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ph, vv, st.o[db], 0, 0, 0);
  }
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const u32x4_t w = v.r[db >> 1];
    const s16x4_t vv = __builtin_bit_cast(s16x4_t, (db & 1) ? make_uint2(w.z, w.w) : make_uint2(w.x, w.y));
    st.o[db] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pl, vv, st.o[db], 0, 0, 0);
  }
}

// One workgroup's attention: query columns c = (row r0 + c / GQA, head
// kh GQA + c % GQA) for c < NCOL (rows >= r0 + nr are unused columns) over
// positions [16 c0, ctx_max) of one slot's tiled K/V plane of kv head kh;
// column c attends the positions below its own limit (row_pos[row] + 1 when
// row_pos_col is given, else ctx_max).  The four waves take interleaved
// 16-position chunks with their own online softmax and leave their states
// in LDS: sm_m[w][c] (running max, log2 units), sm_l[w][c] (sum of
// exponentials), sm_o[(w NCOL + c) HD + d] (unnormalised weighted sums).
// GUARD: some column may see a chunk with no position it attends.
template <int HD, int GQA, int NCOL, bool GUARD, bool NT = true>
__device__ __forceinline__ void attend_block(const float* __restrict__ q, const bf16_t* __restrict__ kc,
                                             const bf16_t* __restrict__ vc, int ctx_stride, long slot_stride,
                                             int slot, int kh, int r0, int nr, int c0, int ctx_max,
                                             const int32_t* __restrict__ row_pos_col, int nq, float (*sm_m)[16],
                                             float (*sm_l)[16], float* sm_o, int pslot = 0, int lo16 = 0) {
  constexpr int DC = HD / 32;     // k-steps of the S product
  constexpr int DB = HD / 16;     // 16-dim blocks of the O product
  static_assert(NCOL <= 16, "16 query columns per workgroup");
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: the chunk branches stay scalar
  const int g = lane >> 4, c16 = lane & 15;
  const int ri = c16 / GQA, hq = c16 % GQA;           // this lane's query column
  const bool valid = c16 < NCOL && ri < nr;
  const int rr = r0 + (valid ? ri : 0);
  const int ctx = (valid && row_pos_col) ? row_pos_col[rr] + 1 : ctx_max;   // positions the column attends
  const size_t plane = (size_t)slot * slot_stride + (size_t)kh * ctx_stride * HD;
  const __amdgpu_buffer_rsrc_t kr_o = buf_rsrc(kc + plane, (uint32_t)ctx_stride * HD * 2);
  const __amdgpu_buffer_rsrc_t vr_o = buf_rsrc(vc + plane, (uint32_t)ctx_stride * HD * 2);
  // chunks below lo16 come from the prefix plane (slot pslot), the rest from
  // the row's own plane; the chunk index is wave-uniform, so the choice is a
  // scalar select of the buffer descriptor
  const size_t pplane = (size_t)pslot * slot_stride + (size_t)kh * ctx_stride * HD;
  const __amdgpu_buffer_rsrc_t kr_p = buf_rsrc(kc + pplane, (uint32_t)ctx_stride * HD * 2);
  const __amdgpu_buffer_rsrc_t vr_p = buf_rsrc(vc + pplane, (uint32_t)ctx_stride * HD * 2);
  const float scale = 1.4426950408889634f / sqrtf((float)HD);   // log2(e) / sqrt(hd)

  // Wave w owns chunks c0 + w, c0 + w + 4, ... of the stream.  The query is
  // requested first and its first three chunks right after, behind a
  // compiler barrier, so that waiting for the query (the wait counter is in
  // issue order) leaves the chunks in flight.
  const float* qp = q + ((size_t)rr * nq + kh * GQA + (valid ? hq : 0)) * HD + 8 * g;
  float4 qa[DC], qb[DC];
#pragma unroll
  for (int dc = 0; dc < DC; ++dc) {
    qa[dc] = *reinterpret_cast<const float4*>(qp + 32 * dc);
    qb[dc] = *reinterpret_cast<const float4*>(qp + 32 * dc + 4);
  }
  asm volatile("" : : : "memory");
  const int nchunk = ((ctx_max + 15) >> 4) - c0;
  const int nmine = nchunk > wave ? (nchunk - wave + 3) >> 2 : 0;
  auto chunk_at = [&](int i) { return c0 + wave + 4 * min(i, nmine - 1); };
  // Six half-chunk slots, three chunks: the K and V tiles of chunk i live in
  // slots 2 (i % 3) and 2 (i % 3) + 1, and each is refilled with the same
  // tile of chunk i + 3 as soon as it is consumed, so while a chunk is
  // consumed the next two to two and a half chunks are in flight.  Loads are issued
  // without branches: a chunk past the wave's last one is read at an offset
  // beyond the buffer's size, which the buffer range check turns into zeros
  // without a memory access (branches around the loads would make the
  // compiler wait for every load in flight at each join).
  const int past = ctx_stride / 16 + 1;            // a chunk index outside the plane
  auto src = [&](int j) { return j < nmine ? chunk_at(j) : past; };
  auto kr = [&](int c) { return c < lo16 ? kr_p : kr_o; };
  auto vr = [&](int c) { return c < lo16 ? vr_p : vr_o; };
  Half<HD> h0, h1, h2, h3, h4, h5;
  load_half<HD, NT>(h0, kr(src(0)), src(0), lane);
  load_half<HD, NT>(h1, vr(src(0)), src(0), lane);
  load_half<HD, NT>(h2, kr(src(1)), src(1), lane);
  load_half<HD, NT>(h3, vr(src(1)), src(1), lane);
  load_half<HD, NT>(h4, kr(src(2)), src(2), lane);
  load_half<HD, NT>(h5, vr(src(2)), src(2), lane);

  // Q^T operand: column c16, k = dims 32dc + 8g .. +7 (zero for unused columns)
  bf16x8_t qh[DC], ql[DC];
#pragma unroll
  for (int dc = 0; dc < DC; ++dc) {
    const float4 a = qa[dc], b = qb[dc];
    float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = valid ? x[e] : 0.f;
    split8(x, qh[dc], ql[dc]);
  }

  AttnState<HD> st;
  st.m_run = -INFINITY;
  st.l_run = 0.f;
#pragma unroll
  for (int db = 0; db < DB; ++db) st.o[db] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // Chunk j of the wave with its K tile in slot ks and its V tile in vs.
  // The pins keep each refill behind the arithmetic that frees its slot and
  // every wait down to the one tile about to be read (left alone, the
  // compiler sinks loads to their first use and the prefetch disappears).
  auto step = [&](int j, Half<HD>& ks, Half<HD>& vs) {
    const int p0 = 16 * chunk_at(j);
    s16x4_t ph, pl;
    pin_half<HD>(ks);
    attend_scores<HD, GUARD>(st, ks, qh, ql, p0, ctx, scale, g, ph, pl);
    pin_half<HD>(ks);
    load_half<HD, NT>(ks, kr(src(j + 3)), src(j + 3), lane);
    pin_half<HD>(vs);
    attend_values<HD>(st, vs, ph, pl, p0, ctx_max, g);
    pin_half<HD>(vs);
    load_half<HD, NT>(vs, vr(src(j + 3)), src(j + 3), lane);
  };
  // whole groups of three chunks as straight-line code, then the last < 3
  int i = 0;
  for (; i + 3 <= nmine; i += 3) {
    step(i, h0, h1);
    step(i + 1, h2, h3);
    step(i + 2, h4, h5);
  }
  if (i < nmine) {
    step(i, h0, h1);
    if (i + 1 < nmine) step(i + 1, h2, h3);
  }

  float l_run = st.l_run;
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  if (lane < 16) {
    sm_m[wave][lane] = st.m_run;
    sm_l[wave][lane] = l_run;
  }
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int h = 4 * g + i;
      if (h < NCOL) sm_o[(wave * NCOL + h) * HD + db * 16 + c16] = st.o[db][i];
    }
  __syncthreads();
}

// Column c, dim d of the four waves' states: the running max M over the
// waves, and the weighted sum and exponential sum rescaled to it (M = -inf
// and zero sums when no wave saw a position).
template <int HD, int NCOL>
__device__ __forceinline__ void waves_merged(const float (*sm_m)[16], const float (*sm_l)[16], const float* sm_o,
                                             int c, int d, float& M, float& num, float& den) {
  M = sm_m[0][c];
#pragma unroll
  for (int w = 1; w < 4; ++w) M = fmaxf(M, sm_m[w][c]);
  num = 0.f;
  den = 0.f;
  if (M == -INFINITY) return;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float f = exp2f(sm_m[w][c] - M);
    num += sm_o[(w * NCOL + c) * HD + d] * f;
    den += sm_l[w][c] * f;
  }
}

// Workgroup (kv head, block of query rows).  Decode (ROWS = 1): one row per
// workgroup, query columns = the GQA heads of the group.  Prompt rows (ROWS =
// 16 / GQA): ROWS consecutive rows of one prompt share the workgroup, each
// column with its own causal limit; the workgroup streams the positions its
// last row attends, so a prompt's K/V is read once per ROWS rows rather than
// once per row.  Row groups of at most 16 rows are split over sub_per_grp
// workgroups of ROWS rows.
template <int HD, int GQA, int ROWS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void attn_mfma_kernel(
    const float* __restrict__ q, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    int ctx_stride, long slot_stride, const int32_t* __restrict__ row_slot,
    const int32_t* __restrict__ row_pos, const int32_t* __restrict__ row_done,
    const int32_t* __restrict__ grp_row0, const int32_t* __restrict__ grp_n, int sub_per_grp,
    bf16_t* __restrict__ out, int nq) {
  constexpr int NCOL = GQA * ROWS;
  __shared__ float sm_m[4][16];
  __shared__ float sm_l[4][16];
  __shared__ float sm_o[4 * NCOL * HD];

  const int kh = blockIdx.x, tid = threadIdx.x;
  int r0 = blockIdx.y, nr = 1;
  if (ROWS > 1) {
    const int grp = blockIdx.y / sub_per_grp, sub = blockIdx.y % sub_per_grp;
    r0 = grp_row0[grp] + sub * ROWS;
    nr = min(ROWS, grp_n[grp] - sub * ROWS);
    if (nr <= 0) return;
  }
  const int col0 = kh * GQA * HD;
  if (ROWS == 1 && row_done && row_done[r0]) {
    bf16_t* orow = out + (size_t)r0 * 2 * nq * HD;     // split-format activation row
    for (int e = tid; e < GQA * HD; e += 256) split_store(orow, col0 + e, 0.f);
    return;
  }
  attend_block<HD, GQA, NCOL, (ROWS > 1)>(q, kc, vc, ctx_stride, slot_stride, row_slot[r0], kh, r0, nr, 0,
                                          row_pos[r0 + nr - 1] + 1, ROWS > 1 ? row_pos : nullptr, nq, sm_m, sm_l,
                                          sm_o);
  for (int e = tid; e < NCOL * HD; e += 256) {
    const int c = e / HD, d = e % HD;
    if (c / GQA >= nr) continue;
    float M, num, den;
    waves_merged<HD, NCOL>(sm_m, sm_l, sm_o, c, d, M, num, den);
    bf16_t* orow = out + (size_t)(r0 + c / GQA) * 2 * nq * HD;
    split_store(orow, col0 + (c % GQA) * HD + d, num / den);
  }
}

// Decode rows whose prompt prefix is shared, one workgroup per (kv head,
// row) and no exchange between workgroups: the row streams positions [0, lo)
// from the plane of the prompt's first sequence (pfx_slot) and [lo, pos] from
// its own.  The G rows of a prompt are consecutive in the grid, so for each
// kv head they run side by side on one XCD and read the prefix through its L2.
template <int HD, int GQA, bool NT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void attn_rows_kernel(
    const float* __restrict__ q, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    int ctx_stride, long slot_stride, const int32_t* __restrict__ row_slot,
    const int32_t* __restrict__ row_pos, const int32_t* __restrict__ row_done,
    const int32_t* __restrict__ row_lo, const int32_t* __restrict__ pfx_slot, bf16_t* __restrict__ out, int nq) {
  __shared__ float sm_m[4][16];
  __shared__ float sm_l[4][16];
  __shared__ float sm_o[4 * GQA * HD];
  const int kh = blockIdx.x, r = blockIdx.y, tid = threadIdx.x;
  const int col0 = kh * GQA * HD;
  bf16_t* orow = out + (size_t)r * 2 * nq * HD;    // split-format activation row
  if (row_done[r]) {
    for (int e = tid; e < GQA * HD; e += 256) split_store(orow, col0 + e, 0.f);
    return;
  }
  const int lo = row_lo[r];
  attend_block<HD, GQA, GQA, false, NT>(q, kc, vc, ctx_stride, slot_stride, row_slot[r], kh, r, 1, 0,
                                        row_pos[r] + 1, nullptr, nq, sm_m, sm_l, sm_o, lo > 0 ? pfx_slot[r] : 0,
                                        lo >> 4);
  for (int e = tid; e < GQA * HD; e += 256) {
    float M, num, den;
    waves_merged<HD, GQA>(sm_m, sm_l, sm_o, e / HD, e % HD, M, num, den);
    split_store(orow, col0 + e, num / den);
  }
}

template <typename KT, bool SPLIT>
__global__ __launch_bounds__(128) void attn_valu_kernel(
    const float* __restrict__ q, const KT* __restrict__ kc, const KT* __restrict__ vc, int hd,
    int ctx_stride, long slot_stride, const int32_t* __restrict__ row_slot,
    const int32_t* __restrict__ row_pos, const int32_t* __restrict__ row_done, void* __restrict__ out,
    int nq, int nkv) {
  __shared__ float sq[128];
  __shared__ float sp[128];
  __shared__ float red[2];
  const int h = blockIdx.x, r = blockIdx.y, tid = threadIdx.x;
  const int width = nq * hd;
  if (row_done && row_done[r]) {
    if (tid < hd) act_store<SPLIT>(out, r, width, h * hd + tid, 0.f);
    return;
  }
  const int kh = h / (nq / nkv);
  const int slot = row_slot[r];
  const int ctx = row_pos[r] + 1;
  const KT* kbase = kc + (size_t)slot * slot_stride + (size_t)kh * ctx_stride * hd;
  const KT* vbase = vc + (size_t)slot * slot_stride + (size_t)kh * ctx_stride * hd;
  if (tid < hd) sq[tid] = q[((size_t)r * nq + h) * hd + tid];
  __syncthreads();
  const float scale = 1.f / sqrtf((float)hd);
  float m_run = -INFINITY, l_run = 0.f, o = 0.f;
  for (int p0 = 0; p0 < ctx; p0 += 128) {
    const int p = p0 + tid;
    float s = -INFINITY;
    if (p < ctx) {
      float acc = 0.f;
      for (int d = 0; d < hd; ++d) acc += sq[d] * ld(kbase + kv_k_index(p, d, hd));
      s = acc * scale;
    }
    float mx = wave_max(s);
    if ((tid & 63) == 0) red[tid >> 6] = mx;
    __syncthreads();
    mx = fmaxf(red[0], red[1]);
    const float m_new = fmaxf(m_run, mx);
    const float alpha = expf(m_run - m_new);
    const float e = p < ctx ? expf(s - m_new) : 0.f;
    sp[tid] = e;
    __syncthreads();
    float ls = wave_sum(e);
    __syncthreads();
    if ((tid & 63) == 0) red[tid >> 6] = ls;
    __syncthreads();
    ls = red[0] + red[1];
    l_run = l_run * alpha + ls;
    if (tid < hd) {
      const int n = min(128, ctx - p0);
      float acc = 0.f;
      for (int t = 0; t < n; ++t) acc += sp[t] * ld(vbase + kv_v_index(p0 + t, tid, hd));
      o = o * alpha + acc;
    }
    m_run = m_new;
    __syncthreads();
  }
  if (tid < hd) act_store<SPLIT>(out, r, width, h * hd + tid, o / l_run);
}

template <int HD, int GQA>
hipError_t run_mfma(const AttnArgs& a, hipStream_t st) {
  constexpr int ROWS = 16 / GQA;
  constexpr int RB = ROWS > 1 ? ROWS : 1;
  const bf16_t* kc = (const bf16_t*)a.cache.k;
  const bf16_t* vc = (const bf16_t*)a.cache.v;
  if (ROWS > 1 && a.grp_row0) {         // prompt rows
    hipLaunchKernelGGL((attn_mfma_kernel<HD, GQA, RB>), dim3(a.nkv, a.n_groups * (16 / RB)), dim3(256), 0, st, a.q,
                       kc, vc, a.cache.ctx_stride, a.cache.slot_stride, a.row_slot, a.row_pos, a.row_done, a.grp_row0,
                       a.grp_n, 16 / RB, (bf16_t*)a.out, a.nq);
    return hipGetLastError();
  }
  if (a.row_lo) {                       // decode rows with a shared prompt prefix
    if (!a.row_done || !a.pfx_slot) return hipErrorInvalidValue;
    hipLaunchKernelGGL((attn_rows_kernel<HD, GQA, true>), dim3(a.nkv, a.R), dim3(256), 0, st, a.q, kc, vc,
                       a.cache.ctx_stride, a.cache.slot_stride, a.row_slot, a.row_pos, a.row_done, a.row_lo,
                       a.pfx_slot, (bf16_t*)a.out, a.nq);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((attn_mfma_kernel<HD, GQA, 1>), dim3(a.nkv, a.R), dim3(256), 0, st, a.q, kc, vc,
                     a.cache.ctx_stride, a.cache.slot_stride, a.row_slot, a.row_pos, a.row_done,
                     (const int32_t*)nullptr, (const int32_t*)nullptr, 1, (bf16_t*)a.out, a.nq);
  return hipGetLastError();
}

template <int HD>
hipError_t dispatch_gqa(const AttnArgs& a, int gqa, hipStream_t st) {
  switch (gqa) {
    case 1: return run_mfma<HD, 1>(a, st);
    case 2: return run_mfma<HD, 2>(a, st);
    case 4: return run_mfma<HD, 4>(a, st);
    case 8: return run_mfma<HD, 8>(a, st);
    case 16: return run_mfma<HD, 16>(a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

bool attention_has_mfma(int dt, int hd, int gqa) {
  return dt == DT_BF16 && (hd == 64 || hd == 128) && (gqa == 1 || gqa == 2 || gqa == 4 || gqa == 8 || gqa == 16);
}

bool attention_shares_prefix(int dt, int hd, int gqa) { return attention_has_mfma(dt, hd, gqa); }

hipError_t launch_attention(const AttnArgs& a, hipStream_t st) {
  if (a.R <= 0) return hipSuccess;
  const int gqa = a.nq / a.nkv;
  if (attention_has_mfma(a.dt, a.hd, gqa)) {
    if (a.hd == 64) return dispatch_gqa<64>(a, gqa, st);
    return dispatch_gqa<128>(a, gqa, st);
  }
  if (a.hd > 128) return hipErrorInvalidValue;
  if (a.dt == DT_BF16)
    hipLaunchKernelGGL((attn_valu_kernel<bf16_t, true>), dim3(a.nq, a.R), dim3(128), 0, st, a.q,
                       (const bf16_t*)a.cache.k, (const bf16_t*)a.cache.v, a.hd, a.cache.ctx_stride,
                       a.cache.slot_stride, a.row_slot, a.row_pos, a.row_done, a.out, a.nq, a.nkv);
  else
    hipLaunchKernelGGL((attn_valu_kernel<float, false>), dim3(a.nq, a.R), dim3(128), 0, st, a.q,
                       (const float*)a.cache.k, (const float*)a.cache.v, a.hd, a.cache.ctx_stride,
                       a.cache.slot_stride, a.row_slot, a.row_pos, a.row_done, a.out, a.nq, a.nkv);
  return hipGetLastError();
}

}  // namespace tandem
