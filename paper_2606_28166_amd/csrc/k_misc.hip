// Row-wise kernels of the tandem step: embedding + RMSNorm, residual +
// RMSNorm, QKV post-processing with the KV append, sampling, the handoff
// rule, prompt-KV replication and per-sequence state set-up.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace tandem {

namespace {

constexpr int kNT = 256;
constexpr int kSplitMaxDev = 16;   // split-K slices a consumer sums (>= the host's cap)

// ------------------------------------------------------------------ norms
// One workgroup per row; each thread owns float4 groups of the row.  All
// split-K partial loads of a group are issued before any is summed (fixed
// order s = 0..S-1), so a row costs one memory round trip, not S.
constexpr int kMaxV4 = 8;          // d_model <= 8192

template <int FMT>
__device__ __forceinline__ void norm_store(void* x, int r, int d, int i4, float4 v, float rs, const float* gain) {
  const float4 gg = *reinterpret_cast<const float4*>(gain + 4 * i4);
  const float y[4] = {v.x * rs * gg.x, v.y * rs * gg.y, v.z * rs * gg.z, v.w * rs * gg.w};
  if (FMT == ACT_F16) {
    const uint2 w = make_uint2((uint32_t)f2h(y[0]) | ((uint32_t)f2h(y[1]) << 16),
                               (uint32_t)f2h(y[2]) | ((uint32_t)f2h(y[3]) << 16));
    reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(x) + (size_t)r * d)[i4] = w;
    return;
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) act_store<FMT == ACT_SPLIT>(x, r, d, 4 * i4 + e, y[e]);
}

template <typename WT, bool SPLIT>
__global__ __launch_bounds__(kNT) void embed_norm_kernel(const int32_t* __restrict__ tok,
                                                         const WT* __restrict__ E, int d,
                                                         const float* __restrict__ gain, float eps,
                                                         float* __restrict__ h, void* __restrict__ x) {
  __shared__ float red[kNT / 64];
  const int r = blockIdx.x, tid = threadIdx.x;
  const WT* e = E + (size_t)tok[r] * d;
  const int n4 = d / 4;
  float4 v[kMaxV4];
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < kMaxV4; ++k) {
    const int i4 = tid + k * kNT;
    v[k] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (i4 < n4) {
      v[k] = make_float4(ld(e + 4 * i4), ld(e + 4 * i4 + 1), ld(e + 4 * i4 + 2), ld(e + 4 * i4 + 3));
      ss += v[k].x * v[k].x + v[k].y * v[k].y + v[k].z * v[k].z + v[k].w * v[k].w;
    }
  }
  const float tot = block_sum<kNT>(ss, red);
  const float rs = 1.f / sqrtf(tot / (float)d + eps);
#pragma unroll
  for (int k = 0; k < kMaxV4; ++k) {
    const int i4 = tid + k * kNT;
    if (i4 < n4) {
      reinterpret_cast<float4*>(h + (size_t)r * d)[i4] = v[k];
      norm_store<SPLIT ? ACT_SPLIT : ACT_F32>(x, r, d, i4, v[k], rs, gain);
    }
  }
}

// At most 64 VGPRs (eight waves per SIMD): a workgroup then fits on a
// compute unit beside two decode-attention waves per SIMD, so the norm that
// follows a projection starts while the other model's attention still holds
// the compute units.  The summed row waits in LDS for the normalisation.
template <int FMT>
__global__ __launch_bounds__(kNT) __attribute__((amdgpu_waves_per_eu(8))) void resid_norm_kernel(
    const float* __restrict__ ws, int S, long ws_stride, float* __restrict__ h, const float* __restrict__ gain,
    float eps, void* __restrict__ x, int d) {
  __shared__ float red[kNT / 64];
  extern __shared__ float4 row[];            // d / 4 entries (launch-sized)
  const int r = blockIdx.x, tid = threadIdx.x;
  const int n4 = d / 4;
  float4* hrow = reinterpret_cast<float4*>(h + (size_t)r * d);
  float ss = 0.f;
  for (int i4 = tid; i4 < n4; i4 += kNT) {
    float4 a = hrow[i4];
    const float4* pp = reinterpret_cast<const float4*>(ws + (size_t)r * d) + i4;
    // fixed order s = 0 .. S-1, eight partial loads in flight
    for (int s0 = 0; s0 < S; s0 += 8) {
      float4 p[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (s0 + u < S) p[u] = pp[(s0 + u) * (ws_stride / 4)];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (s0 + u < S) { a.x += p[u].x; a.y += p[u].y; a.z += p[u].z; a.w += p[u].w; }
    }
    row[i4] = a;
    ss += a.x * a.x + a.y * a.y + a.z * a.z + a.w * a.w;
  }
  const float tot = block_sum<kNT>(ss, red);
  const float rs = 1.f / sqrtf(tot / (float)d + eps);
  for (int i4 = tid; i4 < n4; i4 += kNT) {
    const float4 a = row[i4];
    hrow[i4] = a;
    norm_store<FMT>(x, r, d, i4, a, rs, gain);
  }
}

// ------------------------------------------------------------ SwiGLU finish
// One thread per 8 consecutive outputs of a row (one split-format piece).
__global__ __launch_bounds__(kNT) void swiglu_finish_kernel(const float* __restrict__ ws, int S, long ws_stride,
                                                            int M, int ffn, int interleaved, int f16_out,
                                                            bf16_t* __restrict__ out) {
  const long e = (long)blockIdx.x * kNT + threadIdx.x;
  const int np = ffn / 8;
  if (e >= (long)M * np) return;
  const int m = (int)(e / np), p = (int)(e % np);
  float g[8], u[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) g[i] = u[i] = 0.f;
  // gate and up columns of outputs 8 p .. 8 p + 7
  const int gcol = interleaved ? 32 * (p >> 1) + 8 * (p & 1) : 8 * p;
  const int ucol = interleaved ? gcol + 16 : 8 * p + ffn;
  const float* row = ws + (size_t)m * 2 * ffn;
#pragma unroll
  for (int s = 0; s < kSplitMaxDev; ++s)
    if (s < S) {
      const float4* gp = reinterpret_cast<const float4*>(row + s * ws_stride + gcol);
      const float4* up = reinterpret_cast<const float4*>(row + s * ws_stride + ucol);
      const float4 g0 = gp[0], g1 = gp[1], u0 = up[0], u1 = up[1];
      g[0] += g0.x; g[1] += g0.y; g[2] += g0.z; g[3] += g0.w;
      g[4] += g1.x; g[5] += g1.y; g[6] += g1.z; g[7] += g1.w;
      u[0] += u0.x; u[1] += u0.y; u[2] += u0.z; u[3] += u0.w;
      u[4] += u1.x; u[5] += u1.y; u[6] += u1.z; u[7] += u1.w;
    }
  uint32_t hw[4], lw[4];
  if (f16_out) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float y0 = g[2 * i] / (1.f + expf(-g[2 * i])) * u[2 * i];
      const float y1 = g[2 * i + 1] / (1.f + expf(-g[2 * i + 1])) * u[2 * i + 1];
      hw[i] = (uint32_t)f2h(y0) | ((uint32_t)f2h(y1) << 16);
    }
    reinterpret_cast<uint4*>(out + (size_t)m * ffn)[p] = make_uint4(hw[0], hw[1], hw[2], hw[3]);
    return;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float y0 = g[2 * i] / (1.f + expf(-g[2 * i])) * u[2 * i];
    const float y1 = g[2 * i + 1] / (1.f + expf(-g[2 * i + 1])) * u[2 * i + 1];
    const bf16_t h0 = f2bf(y0), h1 = f2bf(y1);
    hw[i] = (uint32_t)h0 | ((uint32_t)h1 << 16);
    lw[i] = (uint32_t)f2bf(y0 - bf2f(h0)) | ((uint32_t)f2bf(y1 - bf2f(h1)) << 16);
  }
  uint4* o = reinterpret_cast<uint4*>(out + (size_t)m * 2 * ffn + 16 * p);
  o[0] = make_uint4(hw[0], hw[1], hw[2], hw[3]);
  o[1] = make_uint4(lw[0], lw[1], lw[2], lw[3]);
}


// ------------------------------------------------------------ qkv post
// One wave per head of one row (q heads, then k heads, then v heads; four
// heads per workgroup).  Sums the head's split-K partials, applies the
// optional per-head q/k RMSNorm and the NeoX rotary embedding (lane i
// rotates the pair (i, i + hd/2)), writes q, and appends k and v at the
// row's (slot, pos) of the tiled cache.
template <typename KT>
__global__ __launch_bounds__(kNT) void qkv_post_kernel(
    const float* __restrict__ ws, int S, long ws_stride, int nq, int nkv, int hd,
    const float* __restrict__ q_norm, const float* __restrict__ k_norm, float eps,
    const float2* __restrict__ rope, const int32_t* __restrict__ row_slot,
    const int32_t* __restrict__ row_pos, const int32_t* __restrict__ row_done,
    float* __restrict__ q_out, KT* __restrict__ kc, KT* __restrict__ vc, int ctx_stride, long slot_stride) {
  const int r = blockIdx.x, lane = threadIdx.x & 63;
  const int nh = nq + 2 * nkv;
  const int head = blockIdx.y * (kNT / 64) + (threadIdx.x >> 6);
  if (head >= nh) return;
  if (row_done && row_done[r]) return;
  const int half = hd / 2;
  const bool act = lane < half;
  const size_t base = ((size_t)r * nh + head) * hd;
  float x1 = 0.f, x2 = 0.f;
  if (act) {
    float a1[kSplitMaxDev], a2[kSplitMaxDev];
#pragma unroll
    for (int s = 0; s < kSplitMaxDev; ++s)
      if (s < S) {
        a1[s] = ws[s * ws_stride + base + lane];
        a2[s] = ws[s * ws_stride + base + lane + half];
      }
#pragma unroll
    for (int s = 0; s < kSplitMaxDev; ++s)
      if (s < S) {
        x1 += a1[s];
        x2 += a2[s];
      }
  }
  const int slot = row_slot[r], pos = row_pos[r];
  if (head >= nq + nkv) {                      // v head: stored as is
    KT* vo = vc + (size_t)slot * slot_stride + (size_t)(head - nq - nkv) * ctx_stride * hd;
    if (act) {
      st(vo + kv_v_index(pos, lane, hd), x1);
      st(vo + kv_v_index(pos, lane + half, hd), x2);
    }
    return;
  }
  const bool isq = head < nq;
  const float* gn = isq ? q_norm : k_norm;
  if (gn) {
    const float ss = wave_sum(x1 * x1 + x2 * x2);
    const float rs = 1.f / sqrtf(ss / (float)hd + eps);
    if (act) {
      x1 *= rs * gn[lane];
      x2 *= rs * gn[lane + half];
    }
  }
  if (act) {
    const float2 cs = rope[(size_t)pos * half + lane];
    const float y1 = x1 * cs.x - x2 * cs.y;
    const float y2 = x2 * cs.x + x1 * cs.y;
    if (isq) {
      float* qo = q_out + ((size_t)r * nq + head) * hd;
      qo[lane] = y1;
      qo[lane + half] = y2;
    } else {
      KT* ko = kc + (size_t)slot * slot_stride + (size_t)(head - nq) * ctx_stride * hd;
      st(ko + kv_k_index(pos, lane, hd), y1);
      st(ko + kv_k_index(pos, lane + half, hd), y2);
    }
  }
}

__global__ void rope_table_kernel(double theta, int hd, int n_pos, float2* __restrict__ out) {
  const int half = hd / 2;
  const long n = (long)n_pos * half;
  for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < n; e += (long)gridDim.x * blockDim.x) {
    const int p = (int)(e / half), i = (int)(e % half);
    const double inv = pow(theta, -2.0 * i / (double)hd);
    double s, c;
    sincos((double)p * inv, &s, &c);
    out[e] = make_float2((float)c, (float)s);
  }
}

// --------------------------------------------------------------- sampling

// Per (chunk of the vocabulary, row): online log-sum-exp of the senior's
// scores and the top-2 of the owner's Gumbel-perturbed scores.
__global__ __launch_bounds__(kNT) void sample_partials_kernel(SampleArgs a) {
  __shared__ float sm[kNT / 64][5];
  const int ch = blockIdx.x, r = blockIdx.y, tid = threadIdx.x;
  const int s = a.act[r];
  if (a.done[s]) return;
  const int tt = a.t[s];
  const bool own_sen = a.owner[s] != 0;
  const float* zs = a.z_sen + (size_t)r * a.V;
  const float* zj = a.z_jun + (size_t)r * a.V;
  const int v0 = ch * a.chunk, v1 = min(a.V, v0 + a.chunk);
  float ms = -INFINITY, ls = 0.f;
  Top2 top{-INFINITY, 0x7FFFFFFF, -INFINITY};
  for (int base = v0 + tid * 4; base < v1; base += kNT * 4) {
    const u32x4 ph = philox4x32_10(u32x4{(uint32_t)(base >> 2), (uint32_t)tt, (uint32_t)s, 0u}, a.key0, a.key1);
    const uint32_t w[4] = {ph.x, ph.y, ph.z, ph.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int v = base + e;
      if (v < v1) {
        const float sv = (zs[v] + (v == a.eos_id ? a.eos_bias_sen : 0.f)) / a.temp;
        if (sv > ms) { ls = ls * fast_exp(ms - sv) + 1.f; ms = sv; }
        else ls += fast_exp(sv - ms);
        const float so = own_sen ? sv : (zj[v] + (v == a.eos_id ? a.eos_bias_jun : 0.f)) / a.temp;
        const float val = so + gumbel_fast(w[e]);
        top = merge_top2(top, Top2{val, v, -INFINITY});
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(ms, o, 64), l2 = __shfl_xor(ls, o, 64);
    merge_lse(ms, ls, m2, l2);
    Top2 B{__shfl_xor(top.b, o, 64), __shfl_xor(top.i, o, 64), __shfl_xor(top.s, o, 64)};
    top = merge_top2(top, B);
  }
  const int lane = tid & 63, wave = tid >> 6;
  if (lane == 0) {
    sm[wave][0] = ms; sm[wave][1] = ls; sm[wave][2] = top.b;
    sm[wave][3] = __int_as_float(top.i); sm[wave][4] = top.s;
  }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < kNT / 64; ++w) {
      merge_lse(ms, ls, sm[w][0], sm[w][1]);
      top = merge_top2(top, Top2{sm[w][2], __float_as_int(sm[w][3]), sm[w][4]});
    }
    float* p = a.partials + ((size_t)r * gridDim.x + ch) * 5;
    p[0] = ms; p[1] = ls; p[2] = top.b; p[3] = __int_as_float(top.i); p[4] = top.s;
  }
}

// ------------------------------------------------- dual-distribution scores
// Block-wide merge of (max, sum of e^(x - max)) pairs through the waves.
__device__ __forceinline__ void block_lse(float& m, float& l, float (*sm)[2]) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(m, o, 64), l2 = __shfl_xor(l, o, 64);
    merge_lse(m, l, m2, l2);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) { sm[wave][0] = m; sm[wave][1] = l; }
  __syncthreads();
  m = sm[0][0]; l = sm[0][1];
  for (int w = 1; w < kNT / 64; ++w) merge_lse(m, l, sm[w][0], sm[w][1]);
}

// One more value x in a running (max m, sum l of e^(v - m)) (hardware exp2).
__device__ __forceinline__ void lse_add(float& m, float& l, float x) {
  if (x > m) {
    l = l * fast_exp(m - x) + 1.f;
    m = x;
  } else {
    l += fast_exp(x - m);
  }
}

// Pass 1, per (chunk, row): online log-sum-exp partials of both models' logits.
__global__ __launch_bounds__(kNT) void score_lse_kernel(ScoreArgs a) {
  __shared__ float sm[kNT / 64][2];
  const int ch = blockIdx.x, r = blockIdx.y, tid = threadIdx.x;
  if (a.row_done[r]) return;
  const int v0 = ch * a.chunk, v1 = min(a.V, v0 + a.chunk);
  const float* zs = a.z_sen + (size_t)r * a.V;
  const float* zj = a.z_jun + (size_t)r * a.V;
  float ms = -INFINITY, ls = 0.f, mj = -INFINITY, lj = 0.f;
  for (int v = v0 + tid; v < v1; v += kNT) {
    lse_add(ms, ls, zs[v]);
    lse_add(mj, lj, zj[v]);
  }
  block_lse(ms, ls, sm);
  block_lse(mj, lj, sm);
  if (tid == 0) {
    float* p = a.lse + ((size_t)r * a.n_chunks + ch) * 4;
    p[0] = ms; p[1] = ls; p[2] = mj; p[3] = lj;
  }
}

// The row's log-partition functions (log sum_v e^z) of both models from the
// pass-1 partials, in a fixed order.
__device__ __forceinline__ void row_logz(const ScoreArgs& a, int r, float& Ls, float& Lj) {
  float ms = -INFINITY, ls = 0.f, mj = -INFINITY, lj = 0.f;
  for (int c = 0; c < a.n_chunks; ++c) {
    const float* p = a.lse + ((size_t)r * a.n_chunks + c) * 4;
    merge_lse(ms, ls, p[0], p[1]);
    merge_lse(mj, lj, p[2], p[3]);
  }
  Ls = ms + logf(ls);
  Lj = mj + logf(lj);
}

// Pass 2, per (chunk, row): sums of min(p_sen, p_jun) and p_sen (log p_sen - log p_jun).
__global__ __launch_bounds__(kNT) void score_sum_kernel(ScoreArgs a) {
  __shared__ float red[kNT / 64];
  __shared__ float logz[2];
  const int ch = blockIdx.x, r = blockIdx.y, tid = threadIdx.x;
  if (a.row_done[r]) return;
  if (tid == 0) row_logz(a, r, logz[0], logz[1]);
  __syncthreads();
  const float Ls = logz[0], Lj = logz[1];
  const int v0 = ch * a.chunk, v1 = min(a.V, v0 + a.chunk);
  const float* zs = a.z_sen + (size_t)r * a.V;
  const float* zj = a.z_jun + (size_t)r * a.V;
  float smin = 0.f, skl = 0.f;
  for (int v = v0 + tid; v < v1; v += kNT) {
    const float lps = zs[v] - Ls, lpj = zj[v] - Lj;
    const float ps = fast_exp(lps), pj = fast_exp(lpj);
    smin += fminf(ps, pj);
    skl += ps * (lps - lpj);
  }
  smin = block_sum<kNT>(smin, red);
  __syncthreads();
  skl = block_sum<kNT>(skl, red);
  if (tid == 0) {
    float* p = a.sums + ((size_t)r * a.n_chunks + ch) * 2;
    p[0] = smin; p[1] = skl;
  }
}

// One wave per row: the chunk sums (lane-strided, then a fixed butterfly)
// and the junior's cross-entropy.
__global__ __launch_bounds__(64) void score_finish_kernel(ScoreArgs a) {
  const int r = blockIdx.x, lane = threadIdx.x;
  if (a.row_done[r]) return;
  float mj = -INFINITY, lj = 0.f, smin = 0.f, skl = 0.f;
  for (int c = lane; c < a.n_chunks; c += 64) {
    const float* p = a.lse + ((size_t)r * a.n_chunks + c) * 4;
    merge_lse(mj, lj, p[2], p[3]);
    const float* q = a.sums + ((size_t)r * a.n_chunks + c) * 2;
    smin += q[0];
    skl += q[1];
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(mj, o, 64), l2 = __shfl_xor(lj, o, 64);
    merge_lse(mj, lj, m2, l2);
    smin += __shfl_xor(smin, o, 64);
    skl += __shfl_xor(skl, o, 64);
  }
  if (lane != 0) return;
  const float Lj = mj + logf(lj);
  const int s = a.act[r];
  int y = a.tok[s];
  y = y < 0 ? 0 : (y >= a.V ? a.V - 1 : y);
  float* o = a.out + (size_t)s * 3;
  o[0] = Lj - a.z_jun[(size_t)r * a.V + y];
  o[1] = smin;
  o[2] = skl;
}

// One wave per row: merge the chunk partials, pick the token, compute the
// senior log-prob, write the outputs and apply the handoff rule.
__global__ __launch_bounds__(64) void sample_finish_kernel(FinishArgs a) {
  const int r = blockIdx.x, lane = threadIdx.x;
  const int s = a.act[r];
  if (a.done[s]) return;
  float ms = -INFINITY, ls = 0.f;
  Top2 top{-INFINITY, 0x7FFFFFFF, -INFINITY};
  if (a.part_sen) {
    // the LM heads' sampling-epilogue partials: log-sum-exp from the
    // senior's, the top two from the owner's
    const bool own_sen = a.owner[s] != 0;
    for (int c = lane; c < a.n_sen; c += 64) {
      const float* p = a.part_sen + ((size_t)r * a.n_sen + c) * 5;
      merge_lse(ms, ls, p[0], p[1]);
      if (own_sen) top = merge_top2(top, Top2{p[2], __float_as_int(p[3]), p[4]});
    }
    if (!own_sen)
      for (int c = lane; c < a.n_jun; c += 64) {
        const float* p = a.part_jun + ((size_t)r * a.n_jun + c) * 5;
        top = merge_top2(top, Top2{p[2], __float_as_int(p[3]), p[4]});
      }
  } else {
    for (int c = lane; c < a.n_chunks; c += 64) {
      const float* p = a.partials + ((size_t)r * a.n_chunks + c) * 5;
      merge_lse(ms, ls, p[0], p[1]);
      top = merge_top2(top, Top2{p[2], __float_as_int(p[3]), p[4]});
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(ms, o, 64), l2 = __shfl_xor(ls, o, 64);
    merge_lse(ms, ls, m2, l2);
    Top2 B{__shfl_xor(top.b, o, 64), __shfl_xor(top.i, o, 64), __shfl_xor(top.s, o, 64)};
    top = merge_top2(top, B);
  }
  // a row whose scores are all NaN never updates the argmax: keep the index in range
  const int y_hat = (top.i >= 0 && top.i < a.V) ? top.i : 0;
  int y = y_hat;
  if (a.forced) {
    const int f = a.forced[s];
    if (f >= 0 && f < a.V) y = f;
  }
  float zy;
  if (a.part_sen) {
    // the senior logit of the appended token from its LM-head input row
    // (fp16) and the bf16 LM-head row: the product the GEMM formed
    const uint16_t* xr = a.x_sen + (size_t)r * a.d;
    const uint16_t* wr = a.w_lm + (size_t)y * a.d;
    float acc = 0.f;
    for (int k = 8 * lane; k < a.d; k += 512) {
      const uint4 xv = *reinterpret_cast<const uint4*>(xr + k);
      const uint4 wv = *reinterpret_cast<const uint4*>(wr + k);
      const uint32_t xw[4] = {xv.x, xv.y, xv.z, xv.w}, ww[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc += (float)__builtin_bit_cast(_Float16, (uint16_t)(xw[e] & 0xFFFFu)) * bf2f((bf16_t)(ww[e] & 0xFFFFu));
        acc += (float)__builtin_bit_cast(_Float16, (uint16_t)(xw[e] >> 16)) * bf2f((bf16_t)(ww[e] >> 16));
      }
    }
    zy = wave_sum(acc);
  }
  if (lane != 0) return;
  if (!a.part_sen) zy = a.z_sen[(size_t)r * a.V + y];
  const float sy = (zy + (y == a.eos_id ? a.eos_bias_sen : 0.f)) / a.temp;
  const float lp = sy - (ms + logf(ls));
  const int tt = a.t[s];
  const int own = a.owner[s];
  const size_t o = (size_t)s * a.ld_out + (tt - 1);
  a.out_tok[o] = y;
  a.out_own[o] = (uint8_t)(own != 0);
  a.out_lp[o] = lp;
  a.out_len[s] = tt;
  if (a.dbg_sampled) a.dbg_sampled[s] = y_hat;
  if (a.dbg_margin) a.dbg_margin[s] = top.b - top.s;
  const bool is_eos = a.eos_id >= 0 && y == a.eos_id;
  if (!is_eos) {
    const bool is_b = a.bnd ? ((a.bnd[y >> 5] >> (y & 31)) & 1u) != 0 : true;
    const bool at_cap = a.cap_k >= 0 && a.c[s] >= a.cap_k;
    if (is_b || at_cap) {
      const u32x4 ph = philox4x32_10(u32x4{0u, (uint32_t)tt, (uint32_t)s, 1u}, a.key0, a.key1);
      const bool fire = (unsigned long long)ph.x < a.thr;
      int nxt = own;
      if (a.mode == 0) nxt = fire ? 1 : 0;
      else if (a.mode == 1) nxt = fire ? 1 - own : own;
      else nxt = 1 - own;
      a.owner[s] = nxt;
      a.c[s] = 0;
    } else {
      a.c[s] += 1;
    }
  }
  if (is_eos || tt >= a.max_new) a.done[s] = 1;
  a.pending[s] = y;
  a.pos[s] += 1;
  a.t[s] = tt + 1;
}

// ----------------------------------------------------- replication / state
template <typename T>
__global__ __launch_bounds__(kNT) void kv_replicate_kernel(T* kc, T* vc, int nkv, int hd, int ctx_stride,
                                                           long layer_stride, long slot_stride, int src,
                                                           int dst0, int p0, int n_pos) {
  const int lk = blockIdx.x;                 // layer * nkv + kv head
  const int layer = lk / nkv, kh = lk % nkv;
  const int dst = dst0 + blockIdx.y;
  const size_t kh_off = (size_t)kh * ctx_stride * hd;
  // positions p0 .. n_pos-1 (p0 a multiple of 16) occupy the whole
  // 16-position chunks that hold them: a contiguous range of each tiled plane
  const long e0 = (long)p0 * hd;
  const long n = (long)((n_pos + 15) >> 4) * 16 * hd;
  const T* ks = kc + layer * layer_stride + (size_t)src * slot_stride + kh_off;
  T* kd = kc + layer * layer_stride + (size_t)dst * slot_stride + kh_off;
  for (long e = e0 + threadIdx.x; e < n; e += kNT) kd[e] = ks[e];
  const T* vs = vc + layer * layer_stride + (size_t)src * slot_stride + kh_off;
  T* vd = vc + layer * layer_stride + (size_t)dst * slot_stride + kh_off;
  for (long e = e0 + threadIdx.x; e < n; e += kNT) vd[e] = vs[e];
}

__global__ void init_state_kernel(InitStateArgs a) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= a.n_seq) return;
  const int j = s / a.G;
  const int P = a.prompt_len[j];
  int tok = a.prompt_tokens[a.prompt_end[j] - 1];
  if (tok < 0 || tok >= a.V) {
    __hip_atomic_store(a.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    tok = 0;
  }
  a.pending[s] = tok;
  a.pos[s] = P - 1;
  a.t[s] = 1;
  a.c[s] = 0;
  a.done[s] = 0;
  a.out_len[s] = 0;
  int own = a.first_owner;
  if (own == 2) {
    const u32x4 ph = philox4x32_10(u32x4{0u, 0u, (uint32_t)s, 1u}, a.key0, a.key1);
    own = ((unsigned long long)ph.x < a.thr) ? 1 : 0;
  }
  a.owner[s] = own;
}

__global__ void count_active_kernel(const int32_t* done, int n, int32_t* out) {
  __shared__ float red[kNT / 64];
  float c = 0.f;
  for (int i = threadIdx.x; i < n; i += kNT) c += done[i] ? 0.f : 1.f;
  c = block_sum<kNT>(c, red);
  if (threadIdx.x == 0) *out = (int32_t)c;
}

// One workgroup of 1024 threads: a count pass, then a write pass in which
// each 1024-id block places its unfinished ids after the running count of
// earlier ones (block prefix sum) and its finished ids after all unfinished.
__global__ __launch_bounds__(1024) void compact_kernel(const int32_t* __restrict__ done, int n,
                                                       int32_t* __restrict__ act, int32_t* __restrict__ n_out) {
  __shared__ int wsum[16];
  __shared__ int base_a, base_d, total_a;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // block-wide exclusive prefix of flag over the 1024 threads; returns the block total
  auto scan = [&](int flag, int* excl) -> int {
    int x = flag;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    int before = 0, tot = 0;
    for (int i = 0; i < 16; ++i) {
      if (i < w) before += wsum[i];
      tot += wsum[i];
    }
    __syncthreads();
    *excl = before + x - flag;
    return tot;
  };
  int cnt = 0;
  for (int b = 0; b < n; b += 1024) {
    const int s = b + tid;
    int ex;
    cnt += scan(s < n && !done[s] ? 1 : 0, &ex);
  }
  if (tid == 0) { total_a = cnt; base_a = 0; base_d = cnt; }
  __syncthreads();
  for (int b = 0; b < n; b += 1024) {
    const int s = b + tid;
    const int alive = s < n && !done[s] ? 1 : 0;
    const int fin = s < n && done[s] ? 1 : 0;
    int ea, ed;
    const int ta = scan(alive, &ea);
    const int td = scan(fin, &ed);
    if (alive) act[base_a + ea] = s;
    if (fin) act[base_d + ed] = s;
    __syncthreads();
    if (tid == 0) { base_a += ta; base_d += td; }
    __syncthreads();
  }
  if (tid == 0) *n_out = total_a;
}

__global__ void gather_rows_kernel(GatherRowsArgs a) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= a.R) return;
  const int s = a.act[r];
  a.row_tok[r] = a.pending[s];
  a.row_slot[r] = a.seq_slot[s];
  a.row_pos[r] = a.pos[s];
  a.row_done[r] = a.done[s];
}

__global__ void scatter_rows_kernel(const float* __restrict__ src, const int32_t* __restrict__ act, int V,
                                    float* __restrict__ dst) {
  const int r = blockIdx.y;
  const float* sp = src + (size_t)r * V;
  float* dp = dst + (size_t)act[r] * V;
  for (int v = blockIdx.x * blockDim.x + threadIdx.x; v < V; v += gridDim.x * blockDim.x) dp[v] = sp[v];
}

// One workgroup per prompt of the chunk.
__global__ __launch_bounds__(kNT) void prefill_rows_kernel(PrefillRowsArgs a) {
  const int j = a.j0 + blockIdx.x;
  const int P = a.prompt_len[j], start = a.prompt_end[j] - P;
  const int rb = a.row_base[j], gb = a.grp_base[j];
  bool bad = false;
  for (int i = threadIdx.x; i < P - 1; i += kNT) {
    const int r = rb + i;
    int tok = a.prompt_tokens[start + i];
    if (tok < 0 || tok >= a.V) {
      bad = true;
      tok = 0;
    }
    a.row_slot[r] = j * a.G;
    a.row_pos[r] = i;
    a.row_tok[r] = tok;
    if ((i & 15) == 0) {
      a.grp_row0[gb + (i >> 4)] = r;
      a.grp_n[gb + (i >> 4)] = min(16, P - 1 - i);
    }
  }
  if (bad) __hip_atomic_store(a.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Gumbel noise of this step, one Philox call per four vocabulary entries.
__global__ __launch_bounds__(kNT) void gumbel_noise_kernel(const int32_t* __restrict__ act,
                                                           const int32_t* __restrict__ t,
                                                           const int32_t* __restrict__ done, int V, uint32_t k0,
                                                           uint32_t k1, float* __restrict__ noise) {
  const int r = blockIdx.y;
  const int s = act[r];
  if (done[s]) return;
  const int q = blockIdx.x * kNT + threadIdx.x;       // entries 4 q .. 4 q + 3
  if (4 * q >= V) return;
  const u32x4 ph = philox4x32_10(u32x4{(uint32_t)q, (uint32_t)t[s], (uint32_t)s, 0u}, k0, k1);
  reinterpret_cast<float4*>(noise + (size_t)r * V)[q] =
      make_float4(gumbel_fast(ph.x), gumbel_fast(ph.y), gumbel_fast(ph.z), gumbel_fast(ph.w));
}

__global__ void iota_kernel(int32_t* __restrict__ dst, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = i;
}

__global__ void prefix_rows_kernel(const int32_t* __restrict__ act, int R, int G,
                                   const int32_t* __restrict__ prompt_len, int32_t* __restrict__ row_lo,
                                   int32_t* __restrict__ pfx_slot) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= R) return;
  const int j = act[r] / G;
  row_lo[r] = (prompt_len[j] - 1) / 16 * 16;
  pfx_slot[r] = j * G;                        // slots follow sequence ids
}

}  // namespace

hipError_t launch_embed_norm(int dt, const int32_t* tok, const void* E, int d, const float* gain,
                             float eps, float* h, void* x, int R, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  if (dt == DT_BF16)
    hipLaunchKernelGGL((embed_norm_kernel<bf16_t, true>), dim3(R), dim3(kNT), 0, st, tok, (const bf16_t*)E, d,
                       gain, eps, h, x);
  else
    hipLaunchKernelGGL((embed_norm_kernel<float, false>), dim3(R), dim3(kNT), 0, st, tok, (const float*)E, d,
                       gain, eps, h, x);
  return hipGetLastError();
}

hipError_t launch_swiglu_finish(const float* ws, int S, long ws_stride, int M, int ffn, bool interleaved, bool f16_out,
                                void* out, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (S > kSplitMaxDev || ffn % (interleaved ? 16 : 8)) return hipErrorInvalidValue;
  const long n = (long)M * (ffn / 8);
  hipLaunchKernelGGL(swiglu_finish_kernel, dim3((unsigned)((n + kNT - 1) / kNT)), dim3(kNT), 0, st, ws, S, ws_stride,
                     M, ffn, interleaved ? 1 : 0, f16_out ? 1 : 0, (bf16_t*)out);
  return hipGetLastError();
}

hipError_t launch_resid_norm(int dt, const float* ws, int S, long ws_stride, float* h, const float* gain,
                             float eps, void* x, int R, int d, bool f16_out, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  if (S > kSplitMaxDev || (f16_out && dt != DT_BF16)) return hipErrorInvalidValue;
  const size_t lds = (size_t)d * 4;           // the summed row
  if (f16_out)
    hipLaunchKernelGGL((resid_norm_kernel<ACT_F16>), dim3(R), dim3(kNT), lds, st, ws, S, ws_stride, h, gain, eps, x, d);
  else if (dt == DT_BF16)
    hipLaunchKernelGGL((resid_norm_kernel<ACT_SPLIT>), dim3(R), dim3(kNT), lds, st, ws, S, ws_stride, h, gain, eps, x, d);
  else
    hipLaunchKernelGGL((resid_norm_kernel<ACT_F32>), dim3(R), dim3(kNT), lds, st, ws, S, ws_stride, h, gain, eps, x, d);
  return hipGetLastError();
}

hipError_t launch_qkv_post(const QkvPostArgs& a, hipStream_t st) {
  if (a.R <= 0) return hipSuccess;
  if (a.S > kSplitMaxDev || a.hd > 128) return hipErrorInvalidValue;
  const dim3 grid(a.R, (a.nq + 2 * a.nkv + kNT / 64 - 1) / (kNT / 64));
  if (a.dt == DT_BF16)
    hipLaunchKernelGGL((qkv_post_kernel<bf16_t>), grid, dim3(kNT), 0, st, a.ws, a.S, a.ws_stride,
                       a.nq, a.nkv, a.hd, a.q_norm, a.k_norm, a.eps, a.rope, a.row_slot, a.row_pos,
                       a.row_done, a.q_out, (bf16_t*)a.cache.k, (bf16_t*)a.cache.v,
                       a.cache.ctx_stride, a.cache.slot_stride);
  else
    hipLaunchKernelGGL((qkv_post_kernel<float>), grid, dim3(kNT), 0, st, a.ws, a.S, a.ws_stride,
                       a.nq, a.nkv, a.hd, a.q_norm, a.k_norm, a.eps, a.rope, a.row_slot, a.row_pos,
                       a.row_done, a.q_out, (float*)a.cache.k, (float*)a.cache.v,
                       a.cache.ctx_stride, a.cache.slot_stride);
  return hipGetLastError();
}

hipError_t launch_rope_table(float theta, int hd, int n_pos, float2* out, hipStream_t st) {
  hipLaunchKernelGGL(rope_table_kernel, dim3(256), dim3(256), 0, st, (double)theta, hd, n_pos, out);
  return hipGetLastError();
}

hipError_t launch_sample_partials(const SampleArgs& a, int n_chunks, hipStream_t st) {
  if (a.R <= 0) return hipSuccess;
  hipLaunchKernelGGL(sample_partials_kernel, dim3(n_chunks, a.R), dim3(kNT), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_score(const ScoreArgs& a, hipStream_t st) {
  if (a.R <= 0) return hipSuccess;
  if (a.chunk < 1 || a.n_chunks < 1 || (long)a.chunk * a.n_chunks < a.V) return hipErrorInvalidValue;
  hipLaunchKernelGGL(score_lse_kernel, dim3(a.n_chunks, a.R), dim3(kNT), 0, st, a);
  hipLaunchKernelGGL(score_sum_kernel, dim3(a.n_chunks, a.R), dim3(kNT), 0, st, a);
  hipLaunchKernelGGL(score_finish_kernel, dim3(a.R), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_sample_finish(const FinishArgs& a, hipStream_t st) {
  if (a.R <= 0) return hipSuccess;
  hipLaunchKernelGGL(sample_finish_kernel, dim3(a.R), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_kv_replicate(int dt, void* kc, void* vc, int n_layers, long layer_stride,
                               long slot_stride, int nkv, int hd, int ctx_stride, int src,
                               int dst0, int n_dst, int p0, int n_pos, hipStream_t st) {
  if (n_dst <= 0 || n_pos <= p0) return hipSuccess;
  if (p0 < 0 || p0 % 16 || n_pos > ctx_stride) return hipErrorInvalidValue;
  dim3 grid(n_layers * nkv, n_dst);
  if (dt == DT_BF16)
    hipLaunchKernelGGL((kv_replicate_kernel<bf16_t>), grid, dim3(kNT), 0, st, (bf16_t*)kc, (bf16_t*)vc,
                       nkv, hd, ctx_stride, layer_stride, slot_stride, src, dst0, p0, n_pos);
  else
    hipLaunchKernelGGL((kv_replicate_kernel<float>), grid, dim3(kNT), 0, st, (float*)kc, (float*)vc,
                       nkv, hd, ctx_stride, layer_stride, slot_stride, src, dst0, p0, n_pos);
  return hipGetLastError();
}

hipError_t launch_init_state(const InitStateArgs& a, hipStream_t st) {
  if (a.n_seq <= 0) return hipSuccess;
  hipLaunchKernelGGL(init_state_kernel, dim3((a.n_seq + 255) / 256), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_count_active(const int32_t* done, int n, int32_t* out, hipStream_t st) {
  hipLaunchKernelGGL(count_active_kernel, dim3(1), dim3(kNT), 0, st, done, n, out);
  return hipGetLastError();
}

hipError_t launch_compact(const int32_t* done, int n, int32_t* act, int32_t* n_active_out, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(compact_kernel, dim3(1), dim3(1024), 0, st, done, n, act, n_active_out);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const GatherRowsArgs& a, hipStream_t st) {
  if (a.R <= 0) return hipSuccess;
  hipLaunchKernelGGL(gather_rows_kernel, dim3((a.R + 255) / 256), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_scatter_rows(const float* src, const int32_t* act, int R, int V, float* dst, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  hipLaunchKernelGGL(scatter_rows_kernel, dim3(std::min((V + 255) / 256, 64), R), dim3(256), 0, st, src, act, V, dst);
  return hipGetLastError();
}

hipError_t launch_prefill_rows(const PrefillRowsArgs& a, hipStream_t st) {
  if (a.n <= 0) return hipSuccess;
  hipLaunchKernelGGL(prefill_rows_kernel, dim3(a.n), dim3(kNT), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gumbel_noise(const int32_t* act, const int32_t* t, const int32_t* done, int R, int V,
                               uint32_t key0, uint32_t key1, float* noise, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  if (V % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(gumbel_noise_kernel, dim3((V / 4 + kNT - 1) / kNT, R), dim3(kNT), 0, st, act, t, done, V, key0,
                     key1, noise);
  return hipGetLastError();
}

hipError_t launch_iota(int32_t* dst, int n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(iota_kernel, dim3((n + 255) / 256), dim3(256), 0, st, dst, n);
  return hipGetLastError();
}

hipError_t launch_prefix_rows(const int32_t* act, int R, int G, const int32_t* prompt_len, int32_t* row_lo,
                              int32_t* pfx_slot, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  hipLaunchKernelGGL(prefix_rows_kernel, dim3((R + 255) / 256), dim3(256), 0, st, act, R, G, prompt_len, row_lo,
                     pfx_slot);
  return hipGetLastError();
}

}  // namespace tandem
