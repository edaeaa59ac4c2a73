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

template <int HD, int GQA>
__global__ __launch_bounds__(256) void attn_mfma_kernel(
    const float* __restrict__ q, const bf16_t* __restrict__ kc, const bf16_t* __restrict__ vc,
    int ctx_stride, long slot_stride, const int32_t* __restrict__ row_slot,
    const int32_t* __restrict__ row_pos, const int32_t* __restrict__ row_done,
    float* __restrict__ out, int nq) {
  constexpr int DC = HD / 32;     // k-steps of the S product
  constexpr int DB = HD / 16;     // 16-dim blocks of the O product
  constexpr int KSEG = HD / 4;    // dims per lane group
  __shared__ float sm_m[4][16];
  __shared__ float sm_l[4][16];
  __shared__ float sm_o[4][GQA][HD];

  const int kh = blockIdx.x, r = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c16 = lane & 15;
  float* orow = out + (size_t)r * nq * HD + (size_t)kh * GQA * HD;
  if (row_done && row_done[r]) {
    for (int e = tid; e < GQA * HD; e += 256) orow[e] = 0.f;
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
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = valid ? qp[8 * dc + e] : 0.f;
      split8(x, qh[dc], ql[dc]);
    }
  }
  const float scale = 1.4426950408889634f / sqrtf((float)HD);   // log2(e) / sqrt(hd)

  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) o[db] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int nchunk = (ctx + 31) >> 5;
  for (int ch = wave; ch < nchunk; ch += 4) {
    const int p0 = ch * 32;
    // keys of the two 16-position blocks (row = position p0 + 16 pb + c16)
    uint4 kf[2][DC];
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      const int p = min(p0 + 16 * pb + c16, ctx - 1);
      const uint4* kp = reinterpret_cast<const uint4*>(kbase + (size_t)p * HD + g * KSEG);
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) kf[pb][dc] = kp[dc];
    }
    // values: dim db*16 + c16, positions p0 + 4g .. +3 and p0 + 16 + 4g .. +3
    uint2 vf[DB][2];
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const bf16_t* vp = vbase + (size_t)(db * 16 + c16) * ctx_stride + p0 + 4 * g;
      vf[db][0] = *reinterpret_cast<const uint2*>(vp);
      vf[db][1] = *reinterpret_cast<const uint2*>(vp + 16);
    }
    // S^T: lane holds positions p0 + 16 pb + 4g + i for head c16
    float s[2][4];
#pragma unroll
    for (int pb = 0; pb < 2; ++pb) {
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        const bf16x8_t kk = __builtin_bit_cast(bf16x8_t, kf[pb][dc]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, qh[dc], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, ql[dc], acc, 0, 0, 0);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int pp = p0 + 16 * pb + 4 * g + i;
        s[pb][i] = pp < ctx ? acc[i] * scale : -INFINITY;
      }
    }
    float mx = fmaxf(fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3])),
                     fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = exp2f(m_run - m_new);
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
    l_run = l_run * alpha + psum;
    m_run = m_new;
    bf16x8_t ph, pl;
    split8(pr, ph, pl);
    // rescale the accumulator rows (heads 4g + i) by their heads' alpha
    float ai[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) ai[i] = __shfl(alpha, 4 * g + i, 64);
    // mask values past the context (stale cache contents must not leak as 0 * inf)
    const int nvalid0 = ctx - (p0 + 4 * g), nvalid1 = ctx - (p0 + 16 + 4 * g);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      uint2 v0 = vf[db][0], v1 = vf[db][1];
      if (nvalid0 < 4) {
        v0.x = nvalid0 <= 0 ? 0u : (nvalid0 == 1 ? (v0.x & 0xFFFFu) : v0.x);
        v0.y = nvalid0 <= 2 ? 0u : (v0.y & 0xFFFFu);
      }
      if (nvalid1 < 4) {
        v1.x = nvalid1 <= 0 ? 0u : (nvalid1 == 1 ? (v1.x & 0xFFFFu) : v1.x);
        v1.y = nvalid1 <= 2 ? 0u : (v1.y & 0xFFFFu);
      }
      const bf16x8_t vv = __builtin_bit_cast(bf16x8_t, make_uint4(v0.x, v0.y, v1.x, v1.y));
#pragma unroll
      for (int i = 0; i < 4; ++i) o[db][i] *= ai[i];
      o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ph, vv, o[db], 0, 0, 0);
      o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pl, vv, o[db], 0, 0, 0);
    }
  }

  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  if (lane < 16) {
    sm_m[wave][lane] = m_run;
    sm_l[wave][lane] = l_run;
  }
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int h = 4 * g + i;
      if (h < GQA) sm_o[wave][h][db * 16 + c16] = o[db][i];
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
    orow[e] = num / den;
  }
}

template <typename KT>
__global__ __launch_bounds__(128) void attn_valu_kernel(
    const float* __restrict__ q, const KT* __restrict__ kc, const KT* __restrict__ vc, int hd,
    int ctx_stride, long slot_stride, const int32_t* __restrict__ row_slot,
    const int32_t* __restrict__ row_pos, const int32_t* __restrict__ row_done, float* __restrict__ out,
    int nq, int nkv) {
  __shared__ float sq[128];
  __shared__ float sp[128];
  __shared__ float red[2];
  const int h = blockIdx.x, r = blockIdx.y, tid = threadIdx.x;
  float* orow = out + ((size_t)r * nq + h) * hd;
  if (row_done && row_done[r]) {
    if (tid < hd) orow[tid] = 0.f;
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
  if (tid < hd) orow[tid] = o / l_run;
}

template <int HD, int GQA>
hipError_t run_mfma(const AttnArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((attn_mfma_kernel<HD, GQA>), dim3(a.nkv, a.R), dim3(256), 0, st, a.q,
                     (const bf16_t*)a.cache.k, (const bf16_t*)a.cache.v, a.cache.ctx_stride,
                     a.cache.slot_stride, a.row_slot, a.row_pos, a.row_done, a.out, a.nq);
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
    hipLaunchKernelGGL((attn_valu_kernel<bf16_t>), dim3(a.nq, a.R), dim3(128), 0, st, a.q,
                       (const bf16_t*)a.cache.k, (const bf16_t*)a.cache.v, a.hd, a.cache.ctx_stride,
                       a.cache.slot_stride, a.row_slot, a.row_pos, a.row_done, a.out, a.nq, a.nkv);
  else
    hipLaunchKernelGGL((attn_valu_kernel<float>), dim3(a.nq, a.R), dim3(128), 0, st, a.q,
                       (const float*)a.cache.k, (const float*)a.cache.v, a.hd, a.cache.ctx_stride,
                       a.cache.slot_stride, a.row_slot, a.row_pos, a.row_done, a.out, a.nq, a.nkv);
  return hipGetLastError();
}

}  // namespace tandem
