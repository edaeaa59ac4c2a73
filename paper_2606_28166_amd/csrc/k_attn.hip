// Grouped-query attention of one new query position per row over that row's
// KV cache (decode), also used for prompt rows (each prompt token attends to
// positions 0..its own position of the prompt's cache).
//
// bf16 path (HD in {64, 128}): one workgroup per (kv head, row); its four
// waves take interleaved 32-position chunks and keep their own online
// softmax, merged through LDS at the end.  Both products run on MFMA
// 16x16x32 bf16:
//   S^T = K . Q^T   A = 16 cached keys x 32 dims, B = 32 dims x 16 query
//                   heads of the group (heads >= G are zero);
//   O  += P . V     A = 16 heads x 32 positions (the softmax weights, which
//                   each lane already holds for exactly the positions its
//                   k-group needs), B = 32 positions x 16 dims read from the
//                   transposed V cache (4 consecutive positions per load).
// The fp32 query and the fp32 softmax weights enter as bf16 high + low parts
// (two MFMAs each), so only the cache itself is bf16.  K/V stream straight
// from HBM into registers in MFMA layout; one load of a kv head's keys serves
// all G query heads of its group.
//
// fp32 path: a plain VALU kernel, one workgroup per (query head, row).
#include "common.h"
#include "kernels.h"

namespace tandem {

namespace {

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

template <int HD>
struct KVChunk {
  uint4 k[2][HD / 32];            // keys: positions p0 + 16 pb + c16, dims of lane group g
  uint2 v[HD / 16][2];            // values: dim db*16 + c16, positions p0 + 4g .. +3 and p0 + 16 + 4g .. +3
};

template <int HD>
__device__ __forceinline__ void load_chunk(KVChunk<HD>& c, const bf16_t* kbase, const bf16_t* vbase, int p0,
                                           int ctx, int ctx_stride, int g, int c16) {
#pragma unroll
  for (int pb = 0; pb < 2; ++pb) {
    const int p = min(p0 + 16 * pb + c16, ctx - 1);
    const uint4* kp = reinterpret_cast<const uint4*>(kbase + (size_t)p * HD + g * (HD / 4));
#pragma unroll
    for (int dc = 0; dc < HD / 32; ++dc) c.k[pb][dc] = kp[dc];
  }
#pragma unroll
  for (int db = 0; db < HD / 16; ++db) {
    const bf16_t* vp = vbase + (size_t)(db * 16 + c16) * ctx_stride + p0 + 4 * g;
    c.v[db][0] = *reinterpret_cast<const uint2*>(vp);
    c.v[db][1] = *reinterpret_cast<const uint2*>(vp + 16);
  }
}

template <int HD, int GQA>
struct AttnState {
  float m_run, l_run;
  f32x4_t o[HD / 16];
};

template <int HD, int GQA>
__device__ __forceinline__ void attend_chunk(AttnState<HD, GQA>& st, const KVChunk<HD>& c, const bf16x8_t* qh,
                                             const bf16x8_t* ql, int p0, int ctx, float scale, int g) {
  constexpr int DC = HD / 32, DB = HD / 16;
  // S^T: lane holds positions p0 + 16 pb + 4g + i for head c16
  float s[2][4];
  // two independent accumulators per position block (hi and lo query parts)
  // so consecutive MFMAs never wait on each other
  f32x4_t acc[2][2];
#pragma unroll
  for (int pb = 0; pb < 2; ++pb) acc[pb][0] = acc[pb][1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int dc = 0; dc < DC; ++dc)
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      const bf16x8_t kk = __builtin_bit_cast(bf16x8_t, c.k[pb][dc]);
      acc[pb][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, qh[dc], acc[pb][0], 0, 0, 0);
      acc[pb][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, ql[dc], acc[pb][1], 0, 0, 0);
    }
#pragma unroll
  for (int pb = 0; pb < 2; ++pb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int pp = p0 + 16 * pb + 4 * g + i;
      s[pb][i] = pp < ctx ? (acc[pb][0][i] + acc[pb][1][i]) * scale : -INFINITY;
    }
  float mx = fmaxf(fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3])),
                   fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  const float m_new = fmaxf(st.m_run, mx);
  const float alpha = exp2f(st.m_run - m_new);
  float pr[8];
  float psum = 0.f;
#pragma unroll
  for (int pb = 0; pb < 2; ++pb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float p = exp2f(s[pb][i] - m_new);
      pr[4 * pb + i] = p;
      psum += p;
    }
  st.l_run = st.l_run * alpha + psum;
  st.m_run = m_new;
  bf16x8_t ph, pl;
  split8(pr, ph, pl);
  // rescale the accumulator rows (heads 4g + i) by their heads' alpha
  float ai[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) ai[i] = __shfl(alpha, 4 * g + i, 64);
  // mask values past the context (stale cache contents must not leak as 0 * inf)
  const int nvalid0 = ctx - (p0 + 4 * g), nvalid1 = ctx - (p0 + 16 + 4 * g);
  bf16x8_t vv[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    uint2 v0 = c.v[db][0], v1 = c.v[db][1];
    if (nvalid0 < 4) {
      v0.x = nvalid0 <= 0 ? 0u : (nvalid0 == 1 ? (v0.x & 0xFFFFu) : v0.x);
      v0.y = nvalid0 <= 2 ? 0u : (v0.y & 0xFFFFu);
    }
    if (nvalid1 < 4) {
      v1.x = nvalid1 <= 0 ? 0u : (nvalid1 == 1 ? (v1.x & 0xFFFFu) : v1.x);
      v1.y = nvalid1 <= 2 ? 0u : (v1.y & 0xFFFFu);
    }
    vv[db] = __builtin_bit_cast(bf16x8_t, make_uint4(v0.x, v0.y, v1.x, v1.y));
#pragma unroll
    for (int i = 0; i < 4; ++i) st.o[db][i] *= ai[i];
  }
  // hi parts over all dim blocks, then lo parts (independent consecutive MFMAs)
#pragma unroll
  for (int db = 0; db < DB; ++db) st.o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph, vv[db], st.o[db], 0, 0, 0);
#pragma unroll
  for (int db = 0; db < DB; ++db) st.o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl, vv[db], st.o[db], 0, 0, 0);
}

template <int HD, int GQA>
__global__ __launch_bounds__(256) void attn_mfma_kernel(
    const float* __restrict__ q, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    int ctx_stride, long slot_stride, const int32_t* __restrict__ row_slot,
    const int32_t* __restrict__ row_pos, const int32_t* __restrict__ row_done,
    bf16_t* __restrict__ out, int nq) {
  constexpr int DC = HD / 32;     // k-steps of the S product
  constexpr int DB = HD / 16;     // 16-dim blocks of the O product
  constexpr int KSEG = HD / 4;    // dims per lane group
  __shared__ float sm_m[4][16];
  __shared__ float sm_l[4][16];
  __shared__ float sm_o[4][GQA][HD];

  const int kh = blockIdx.x, r = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c16 = lane & 15;
  bf16_t* orow = out + (size_t)r * 2 * nq * HD;       // split-format activation row
  const int col0 = kh * GQA * HD;
  if (row_done && row_done[r]) {
    for (int e = tid; e < GQA * HD; e += 256) split_store(orow, col0 + e, 0.f);
    return;
  }
  const int slot = row_slot[r];
  const int ctx = row_pos[r] + 1;
  const bf16_t* kbase = kc + (size_t)slot * slot_stride + (size_t)kh * ctx_stride * HD;
  const bf16_t* vbase = vc + (size_t)slot * slot_stride + (size_t)kh * HD * ctx_stride;

  // Q^T operand: column = query head c16 of this group, k = dims of group g
  bf16x8_t qh[DC], ql[DC];
  {
    const bool valid = c16 < GQA;
    const float* qp = q + ((size_t)r * nq + kh * GQA + (valid ? c16 : 0)) * HD + g * KSEG;
#pragma unroll
    for (int dc = 0; dc < DC; ++dc) {
      const float4 a = *reinterpret_cast<const float4*>(qp + 8 * dc);
      const float4 b = *reinterpret_cast<const float4*>(qp + 8 * dc + 4);
      float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = valid ? x[e] : 0.f;
      split8(x, qh[dc], ql[dc]);
    }
  }
  const float scale = 1.4426950408889634f / sqrtf((float)HD);   // log2(e) / sqrt(hd)

  AttnState<HD, GQA> st;
  st.m_run = -INFINITY;
  st.l_run = 0.f;
#pragma unroll
  for (int db = 0; db < DB; ++db) st.o[db] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // two register buffers: the next chunk of this wave is in flight while the
  // current one is consumed; past the end the current chunk is reloaded (an
  // L2 hit) so every iteration issues the same loads
  const int nchunk = (ctx + 31) >> 5;
  KVChunk<HD> ca, cb;
  if (wave < nchunk) load_chunk<HD>(ca, kbase, vbase, 32 * wave, ctx, ctx_stride, g, c16);
  for (int ch = wave; ch < nchunk; ch += 8) {
    const int nb = ch + 4 < nchunk ? ch + 4 : ch;
    load_chunk<HD>(cb, kbase, vbase, 32 * nb, ctx, ctx_stride, g, c16);
    attend_chunk<HD, GQA>(st, ca, qh, ql, 32 * ch, ctx, scale, g);
    if (ch + 4 >= nchunk) break;
    const int na = ch + 8 < nchunk ? ch + 8 : ch + 4;
    load_chunk<HD>(ca, kbase, vbase, 32 * na, ctx, ctx_stride, g, c16);
    attend_chunk<HD, GQA>(st, cb, qh, ql, 32 * (ch + 4), ctx, scale, g);
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
      if (h < GQA) sm_o[wave][h][db * 16 + c16] = st.o[db][i];
    }
  __syncthreads();
  for (int e = tid; e < GQA * HD; e += 256) {
    const int h = e / HD, d = e % HD;
    float M = sm_m[0][h];
#pragma unroll
    for (int w = 1; w < 4; ++w) M = fmaxf(M, sm_m[w][h]);
    float num = 0.f, den = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float f = exp2f(sm_m[w][h] - M);
      num += sm_o[w][h][d] * f;
      den += sm_l[w][h] * f;
    }
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
  const KT* vbase = vc + (size_t)slot * slot_stride + (size_t)kh * hd * ctx_stride;
  if (tid < hd) sq[tid] = q[((size_t)r * nq + h) * hd + tid];
  __syncthreads();
  const float scale = 1.f / sqrtf((float)hd);
  float m_run = -INFINITY, l_run = 0.f, o = 0.f;
  for (int p0 = 0; p0 < ctx; p0 += 128) {
    const int p = p0 + tid;
    float s = -INFINITY;
    if (p < ctx) {
      float acc = 0.f;
      for (int d = 0; d < hd; ++d) acc += sq[d] * ld(kbase + (size_t)p * hd + d);
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
      for (int t = 0; t < n; ++t) acc += sp[t] * ld(vbase + (size_t)tid * ctx_stride + p0 + t);
      o = o * alpha + acc;
    }
    m_run = m_new;
    __syncthreads();
  }
  if (tid < hd) act_store<SPLIT>(out, r, width, h * hd + tid, o / l_run);
}

template <int HD, int GQA>
hipError_t run_mfma(const AttnArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((attn_mfma_kernel<HD, GQA>), dim3(a.nkv, a.R), dim3(256), 0, st, a.q,
                     (const bf16_t*)a.cache.k, (const bf16_t*)a.cache.v, a.cache.ctx_stride,
                     a.cache.slot_stride, a.row_slot, a.row_pos, a.row_done, (bf16_t*)a.out, a.nq);
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
