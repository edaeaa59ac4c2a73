// Projection GEMMs of the decoder: C = A . W^T with W row-major [out][in],
// A the fp32 activations (normed hidden states, attention output, SwiGLU
// output).
//
// bf16 path (gfx950 MFMA, v_mfma_f32_16x16x32_bf16): a weight-streaming
// kernel.  Each wave owns NB blocks of 16 weight rows and streams them from
// HBM straight into registers, D chunks of 64 k-values ahead.  The activation
// tile (BM rows x 64 k) is staged once per workgroup through LDS, split into
// a bf16 high part and a bf16 low part (x = hi + lo to about 2^-16), and
// every weight fragment meets both: two MFMAs, fp32 accumulation.  The
// activations therefore keep fp32-level precision while the weights stream
// at bf16 width; decode projections are bound by the weight stream, so the
// second MFMA is nearly free.  LDS rows are padded by 16 bytes so the
// MFMA-layout reads are free of bank conflicts.  K may be split over grid.z;
// the partial tiles are summed by the consuming kernel in a fixed order,
// which keeps results bitwise reproducible.
//
// MFMA operand layout used (16x16x32): lane l supplies row/column l % 16 and
// eight k-values of group l / 16; the result lane l holds column l % 16 of
// rows 4 * (l / 16) .. + 3.  Any permutation of k that is the same for both
// operands gives the same dot product, so lane group g takes the contiguous
// k range [16 g, 16 g + 16) of each 64-wide chunk: one 32-byte run per lane.
//
// fp32 path: a plain LDS-tiled VALU kernel (fp32 models and K that is not a
// multiple of 64).
#include "common.h"
#include "kernels.h"

namespace tandem {

namespace {

constexpr int BK = kGemmBK;        // k-values per chunk
constexpr int LDA = BK + 8;        // padded LDS row (elements)

__device__ __forceinline__ float silu(float x) { return x / (1.f + expf(-x)); }

template <int MT, int NB, int EPI, int D>
__global__ __launch_bounds__(256) void gemm_mfma_kernel(
    const float* __restrict__ A, const bf16_t* __restrict__ W, int M, int N, int K, int cps,
    float* __restrict__ out, int ldo, long split_stride) {
  constexpr int BM = 16 * MT;
  constexpr int PIECES = BM * (BK / 4);               // float4 pieces of one A chunk
  constexpr int AITER = (PIECES + 255) / 256;
  __shared__ __attribute__((aligned(16))) bf16_t Ah[BM][LDA];
  __shared__ __attribute__((aligned(16))) bf16_t Al[BM][LDA];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c16 = lane & 15;
  const int m0 = blockIdx.y * BM;
  const int nch = K / BK;
  const int kc0 = blockIdx.z * cps;
  const int nloc = min(cps, nch - kc0);
  if (nloc <= 0) return;

  // weight rows streamed by this lane
  const bf16_t* wrow[NB];
  int ncol[NB];
  if (EPI == EPI_SWIGLU) {
    const int j = blockIdx.x * 64 + wave * 16 + c16;
    ncol[0] = j;
    ncol[1] = j;
    const int jc = min(j, N - 1);
    wrow[0] = W + (size_t)jc * K;
    wrow[1] = W + (size_t)(N + jc) * K;
  } else {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int n = blockIdx.x * (64 * NB) + (wave * NB + nb) * 16 + c16;
      ncol[nb] = n;
      wrow[nb] = W + (size_t)min(n, N - 1) * K;
    }
  }

  u32x4_t wbuf[D][NB][2];
  float4 areg[AITER];

  auto load_w = [&](int it, u32x4_t (&dst)[NB][2]) {
    const size_t off = (size_t)(kc0 + it) * BK + 16 * g;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const u32x4_t* p = reinterpret_cast<const u32x4_t*>(wrow[nb] + off);
      dst[nb][0] = __builtin_nontemporal_load(p);
      dst[nb][1] = __builtin_nontemporal_load(p + 1);
    }
  };
  auto load_a = [&](int it) {
#pragma unroll
    for (int i = 0; i < AITER; ++i) {
      const int piece = tid + 256 * i;
      const int r = piece >> 4, cc = (piece & 15) * 4;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (piece < PIECES && m0 + r < M)
        v = *reinterpret_cast<const float4*>(A + (size_t)(m0 + r) * K + (size_t)(kc0 + it) * BK + cc);
      areg[i] = v;
    }
  };
  auto store_a = [&]() {
#pragma unroll
    for (int i = 0; i < AITER; ++i) {
      const int piece = tid + 256 * i;
      if (piece < PIECES) {
        const int r = piece >> 4, cc = (piece & 15) * 4;
        const float x[4] = {areg[i].x, areg[i].y, areg[i].z, areg[i].w};
        bf16_t hi[4], lo[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          hi[e] = f2bf(x[e]);
          lo[e] = f2bf(x[e] - bf2f(hi[e]));
        }
        *reinterpret_cast<uint2*>(&Ah[r][cc]) =
            make_uint2((uint32_t)hi[0] | ((uint32_t)hi[1] << 16), (uint32_t)hi[2] | ((uint32_t)hi[3] << 16));
        *reinterpret_cast<uint2*>(&Al[r][cc]) =
            make_uint2((uint32_t)lo[0] | ((uint32_t)lo[1] << 16), (uint32_t)lo[2] | ((uint32_t)lo[3] << 16));
      }
    }
  };

  f32x4_t acc[MT][NB];
#pragma unroll
  for (int mb = 0; mb < MT; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  load_a(0);
#pragma unroll
  for (int d = 0; d < D - 1; ++d)
    if (d < nloc) load_w(d, wbuf[d]);

  for (int kk = 0; kk < nloc; kk += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int it = kk + d;
      if (it < nloc) {
        if (it + D - 1 < nloc) load_w(it + D - 1, wbuf[(d + D - 1) % D]);
        __syncthreads();              // every wave is done reading the previous chunk
        store_a();
        __syncthreads();
        if (it + 1 < nloc) load_a(it + 1);
#pragma unroll
        for (int j = 0; j < 2; ++j) {
#pragma unroll
          for (int mb = 0; mb < MT; ++mb) {
            const bf16x8_t ah = *reinterpret_cast<const bf16x8_t*>(&Ah[mb * 16 + c16][16 * g + 8 * j]);
            const bf16x8_t al = *reinterpret_cast<const bf16x8_t*>(&Al[mb * 16 + c16][16 * g + 8 * j]);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
              const bf16x8_t b = __builtin_bit_cast(bf16x8_t, wbuf[d][nb][j]);
              acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, b, acc[mb][nb], 0, 0, 0);
              acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, b, acc[mb][nb], 0, 0, 0);
            }
          }
        }
      }
    }
  }

  // epilogue
#pragma unroll
  for (int mb = 0; mb < MT; ++mb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + mb * 16 + 4 * g + i;
      if (m >= M) continue;
      if (EPI == EPI_SWIGLU) {
        const int j = ncol[0];
        if (j < N) out[(size_t)m * ldo + j] = silu(acc[mb][0][i]) * acc[mb][1][i];
      } else {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int n = ncol[nb];
          if (n < N) out[blockIdx.z * split_stride + (size_t)m * ldo + n] = acc[mb][nb][i];
        }
      }
    }
  }
}

// ---------------------------------------------------------------- VALU path
template <typename WT, int EPI>
__global__ __launch_bounds__(256) void gemm_valu_kernel(
    const float* __restrict__ A, const WT* __restrict__ W, int M, int N, int K, int kper,
    float* __restrict__ out, int ldo, long split_stride) {
  // 32 x 32 output tile, 16 x 16 threads with 2 x 2 outputs each
  constexpr int T = 32;
  constexpr int NW = (EPI == EPI_SWIGLU) ? 2 : 1;
  __shared__ float As[T][T + 1];
  __shared__ float Ws[NW][T][T + 1];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m0 = blockIdx.y * T, n0 = blockIdx.x * T;
  const int kb = blockIdx.z * kper, ke = min(K, kb + kper);
  float acc[NW][2][2] = {};
  for (int k0 = kb; k0 < ke; k0 += T) {
    for (int e = threadIdx.x; e < T * T; e += 256) {
      const int r = e / T, c = e % T;
      const int m = m0 + r, k = k0 + c;
      As[r][c] = (m < M && k < ke) ? A[(size_t)m * K + k] : 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const int n = n0 + r;
        const int row = n + w * N;
        Ws[w][r][c] = (n < N && k < ke) ? ld(W + (size_t)row * K + k) : 0.f;
      }
    }
    __syncthreads();
    for (int kk = 0; kk < T; ++kk) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const float a = As[ty * 2 + i][kk];
#pragma unroll
        for (int w = 0; w < NW; ++w)
#pragma unroll
          for (int jj = 0; jj < 2; ++jj) acc[w][i][jj] += a * Ws[w][tx * 2 + jj][kk];
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      const int m = m0 + ty * 2 + i, n = n0 + tx * 2 + jj;
      if (m >= M || n >= N) continue;
      if (EPI == EPI_SWIGLU)
        out[(size_t)m * ldo + n] = silu(acc[0][i][jj]) * acc[NW - 1][i][jj];
      else
        out[blockIdx.z * split_stride + (size_t)m * ldo + n] = acc[0][i][jj];
    }
}

template <int MT, int NB, int EPI>
hipError_t run_mfma(const GemmArgs& a, int S, int cps, hipStream_t st) {
  constexpr int D = 4;
  const int cols = (EPI == EPI_SWIGLU) ? 64 : 64 * NB;
  dim3 grid((a.N + cols - 1) / cols, (a.M + 16 * MT - 1) / (16 * MT), S);
  hipLaunchKernelGGL((gemm_mfma_kernel<MT, NB, EPI, D>), grid, dim3(256), 0, st, a.A, (const bf16_t*)a.W,
                     a.M, a.N, a.K, cps, a.out, a.ldo, a.split_stride);
  return hipGetLastError();
}

template <int EPI>
hipError_t dispatch_mfma(const GemmArgs& a, int S, int cps, hipStream_t st) {
  const int mt_need = (min(a.M, 128) + 15) / 16;
  constexpr int NB = 2;
  if (mt_need <= 1) return run_mfma<1, NB, EPI>(a, S, cps, st);
  if (mt_need <= 2) return run_mfma<2, NB, EPI>(a, S, cps, st);
  if (mt_need <= 4) return run_mfma<4, NB, EPI>(a, S, cps, st);
  return run_mfma<8, NB, EPI>(a, S, cps, st);
}

template <typename WT>
hipError_t run_valu(const GemmArgs& a, int S, int kper, hipStream_t st) {
  dim3 grid((a.N + 31) / 32, (a.M + 31) / 32, S);
  if (a.epi == EPI_SWIGLU)
    hipLaunchKernelGGL((gemm_valu_kernel<WT, EPI_SWIGLU>), grid, dim3(256), 0, st, a.A, (const WT*)a.W,
                       a.M, a.N, a.K, kper, a.out, a.ldo, a.split_stride);
  else
    hipLaunchKernelGGL((gemm_valu_kernel<WT, EPI_PARTIAL>), grid, dim3(256), 0, st, a.A, (const WT*)a.W,
                       a.M, a.N, a.K, kper, a.out, a.ldo, a.split_stride);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& a, int* splits_used, hipStream_t st) {
  if (a.M <= 0 || a.N <= 0) {
    if (splits_used) *splits_used = 0;
    return hipSuccess;
  }
  int S = a.epi == EPI_PARTIAL ? (a.splits < 1 ? 1 : a.splits) : 1;
  const bool mfma = (a.dt == DT_BF16) && (a.K % BK == 0);
  if (mfma) {
    const int nch = a.K / BK;
    if (S > nch) S = nch;
    const int cps = (nch + S - 1) / S;
    S = (nch + cps - 1) / cps;
    if (splits_used) *splits_used = S;
    switch (a.epi) {
      case EPI_PARTIAL: return dispatch_mfma<EPI_PARTIAL>(a, S, cps, st);
      case EPI_STORE: return dispatch_mfma<EPI_STORE>(a, S, cps, st);
      default: return dispatch_mfma<EPI_SWIGLU>(a, S, cps, st);
    }
  }
  const int nk = (a.K + 31) / 32;
  if (S > nk) S = nk;
  const int kper = ((nk + S - 1) / S) * 32;
  S = (a.K + kper - 1) / kper;
  if (splits_used) *splits_used = S;
  if (a.dt == DT_BF16) return run_valu<bf16_t>(a, S, kper, st);
  return run_valu<float>(a, S, kper, st);
}

}  // namespace tandem
