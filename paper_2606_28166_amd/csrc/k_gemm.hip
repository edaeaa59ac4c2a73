// Projection GEMMs of the decoder: C = A . W^T with W row-major [out][in].
//
// bf16 path (gfx950 MFMA v_mfma_f32_32x32x16_bf16), a streaming kernel for
// skinny (decode) and tall (prefill) A alike:
//   * A holds the activations in split format (per 8 values: 8 bf16 high
//     parts, then 8 bf16 low parts), so every weight fragment meets hi and lo
//     in two MFMAs: fp32-level activations, bf16 weights, fp32 accumulation.
//   * One workgroup computes a BM x BN output tile (BM in {32, 64, 128, 256},
//     BN 128 or 256) over its slice of K, 64 k-values per chunk.  With BM >=
//     128 its 8 waves (two per SIMD, so one issues MFMAs while the other
//     waits on LDS) tile the 32 x 32 MFMA blocks 4 x 2; smaller tiles use 4
//     waves (2 x 2, or 1 x 4 when BM = 32).  The 32 x 32 x 16 shape keeps the matrix cores
//     near their peak with only a few accumulators per wave.
//   * Weight rows and activation rows of each chunk stream into an NS-stage
//     LDS ring with global_load_lds_dwordx4 (no register staging); 16-byte
//     pieces are XOR-swizzled by row so the MFMA-layout reads spread over all
//     banks.  All loads are issued unconditionally (clamped to the last
//     chunk), the reads are explicit ds_read_b128, and the only waits are
//     compile-time vmcnt/lgkmcnt values plus a raw s_barrier: the compiler
//     never sees a memory result it could over-wait for, so NS - 1 chunks
//     stay in flight the whole time.
//   * K may be split over grid.z; the consuming kernel sums the partial
//     tiles in a fixed order, keeping results bitwise reproducible.
//
// MFMA operand layout (32x32x16): lane l supplies row/column l % 32 and eight
// k-values of group l / 32; result element i of lane l is column l % 32 of
// row 8 (i / 4) + 4 (l / 32) + i % 4.  Any permutation of k that is the same
// for both operands gives the same dot product, so lane group g takes the
// k range [32 g, 32 g + 32) of each chunk, 8 values per k-step.
//
// fp32 path: a plain LDS-tiled VALU kernel (fp32 models, K not a multiple of 64).
#include "common.h"
#include "kernels.h"

namespace tandem {

namespace {

constexpr int BK = kGemmBK;        // k-values per chunk

__device__ __forceinline__ float silu(float x) { return x / (1.f + expf(-x)); }

template <int BMT, int BNT, int NST, int NWT = 4, bool A16 = false> struct GemmShape {
  static constexpr int NW = NWT;                      // waves per workgroup (4 or 8)
  static constexpr int BM = BMT;
  static constexpr int BN = BNT;                      // weight rows per tile (128 or 256)
  static constexpr int MB = BM / 32;                  // 32-row blocks
  static constexpr int WM = NW == 8 ? (MB >= 4 ? 4 : MB) : (MB >= 2 ? 2 : 1);   // waves along M
  static constexpr int WN = NW / WM;                  // waves along N
  static constexpr int MBW = MB / WM;                 // 32-row blocks per wave
  static constexpr int NBW = BN / 32 / WN;            // 32-column blocks per wave
  static constexpr int NS = NST;                      // ring stages
  static constexpr int PARTS = A16 ? 1 : 2;           // MFMA operand parts per activation (fp16, or hi + lo)
  static constexpr int RB = BK * 2 * PARTS;           // bytes of one activation row per chunk
  static constexpr int NPC = RB / 16;                 // 16-byte pieces per activation row
  static constexpr int RPI = 64 / NPC;                // activation rows per 1 KB DMA instruction
  static constexpr int ASTAGE = BM * RB;              // bytes of one activation stage
  static constexpr int WSTAGE = BN * BK * 2;          // bytes of one weight stage
  static constexpr int STAGE = ASTAGE + WSTAGE;
  static constexpr int NA = BM / (RPI * NW);          // activation DMA instructions per wave per chunk
  static constexpr int NWD = BN / (8 * NW);           // weight DMA instructions per wave per chunk
  static constexpr int WAIT = (NS - 2) * (NA + NWD);  // vmcnt that leaves NS - 2 chunks in flight
  static constexpr int OUT_COLS = BN / 2;             // SwiGLU output columns per tile
  static_assert(NS * STAGE <= 160 * 1024, "LDS ring exceeds 160 KB");
  static_assert(NA >= 1 && NWD >= 1 && MBW >= 1 && NBW >= 1, "tile too small for the waves");
};

// PK: the weights come from the packed MFMA-fragment copy (pair-interleaved
// for SwiGLU, like the tile rows below) instead of the row-major matrix: one
// 1 KB fragment per DMA instruction, lane-contiguous fragment reads.  The
// k-order inside a chunk then follows the packed layout (lane half g of k-step
// j holds k-group 2 j + g).  A16: fp16 activations against fp16 packed weights
// (PK only).
template <int BMT, int BNT, int NST, int EPI, int NWT, bool PK = false, bool A16 = false>
__global__ __launch_bounds__(64 * NWT) void gemm_mfma_kernel(
    const bf16_t* __restrict__ A, const bf16_t* __restrict__ W, int M, int N, int K, int cps,
    float* __restrict__ out, int ldo, long split_stride) {
  using G = GemmShape<BMT, BNT, NST, NWT, A16>;
  static_assert(PK || !A16, "fp16 activations need the fp16 packed weights");
  constexpr int PARTS = G::PARTS, NPC = G::NPC;
  __shared__ __attribute__((aligned(1024))) unsigned char ring[G::NS * G::STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, c32 = lane & 31;
  const int wm = wave / G::WN, wn = wave % G::WN;
  const int m0 = blockIdx.y * G::BM;
  const int nch = K / BK;
  const int kc0 = blockIdx.z * cps;
  const int nloc = min(cps, nch - kc0);
  if (nloc <= 0) return;

  // Global weight row of tile row t (0..BN-1).  SwiGLU tiles pair gate and up
  // rows inside every 32-row block: rows 32p .. 32p+15 are gate rows
  // j0 + 16p + c, rows 32p+16 .. 32p+31 the matching up rows; other tiles
  // hold BN consecutive rows.
  auto wrow_of = [&](int t) -> int {
    if (EPI == EPI_SWIGLU) {
      const int j = min(blockIdx.x * G::OUT_COLS + 16 * (t >> 5) + (t & 15), N - 1);
      return ((t >> 4) & 1) ? N + j : j;
    }
    return min(blockIdx.x * G::BN + t, N - 1);
  };

  // DMA sources.  Weight stage: instruction i of wave w covers tile rows
  // (BN/NW) w + 8i .. +8 (128 B each); lane -> row (lane >> 3), physical
  // piece lane & 7 holding logical piece (lane & 7) ^ ((row >> 1) & 7).
  // Packed weights: instruction i of wave w moves fragment f = NW i + w of
  // the stage (32-row block f / 4 of the tile, k-step f % 4), 1 KB.
  const bf16_t* wsrc[G::NWD];
  const int kfr = K / 16;                               // fragments per packed 32-row block
#pragma unroll
  for (int i = 0; i < G::NWD; ++i) {
    if (PK) {
      const int f = G::NW * i + wave;
      const int blk = min(blockIdx.x * (G::BN / 32) + f / 4, ((EPI == EPI_SWIGLU ? 2 * N : N) + 31) / 32 - 1);
      wsrc[i] = W + ((size_t)blk * kfr + f % 4) * 512 + lane * 8;
    } else {
      const int t = (G::BN / G::NW) * wave + 8 * i + (lane >> 3);
      const int lp = (lane & 7) ^ ((t >> 1) & 7);
      wsrc[i] = W + (size_t)wrow_of(t) * K + lp * 8;
    }
  }
  // Activation stage: instruction i of wave w covers tile rows RPI (NW i + w) ..
  // +RPI - 1 (a row is NPC 16-byte pieces: split format 8 hi and 8 lo pieces,
  // fp16 8 pieces); physical piece lane % NPC holds logical piece
  // (lane % NPC) ^ (row % NPC).
  const bf16_t* asrc[G::NA];
#pragma unroll
  for (int i = 0; i < G::NA; ++i) {
    const int r = G::RPI * (G::NW * i + wave) + lane / NPC;
    const int lc = (lane % NPC) ^ (r % NPC);
    asrc[i] = A + (size_t)min(m0 + r, M - 1) * PARTS * (size_t)K + lc * 8;
  }
  unsigned char* const ring0 = ring;
  auto issue = [&](int it) {
    const int c = kc0 + min(it, nloc - 1);
    unsigned char* st = ring0 + (it % G::NS) * G::STAGE;
#pragma unroll
    for (int i = 0; i < G::NA; ++i)
      load_lds16(asrc[i] + (size_t)c * PARTS * BK, st + (G::NW * i + wave) * 1024);
#pragma unroll
    for (int i = 0; i < G::NWD; ++i) {
      if (PK) load_lds16_nt(wsrc[i] + (size_t)c * 4 * 512, st + G::ASTAGE + (G::NW * i + wave) * 1024);
      else load_lds16_nt(wsrc[i] + (size_t)c * BK, st + G::ASTAGE + ((G::BN / G::NW) * wave + 8 * i) * 128);
    }
  };

  f32x16_t acc[G::MBW][G::NBW];
#pragma unroll
  for (int mb = 0; mb < G::MBW; ++mb)
#pragma unroll
    for (int nb = 0; nb < G::NBW; ++nb) acc[mb][nb] = f32x16_t{};

  const uint32_t ring_addr = lds_addr_of(ring);
  struct Frags {
    u32x4_t a[G::MBW][PARTS];
    u32x4_t w[G::NBW];
  };
  // fragments of k-step j: k-group q of rows / columns c32 of each block
  // (q = 4 g + j for row-major weights, 2 j + g for packed ones)
  auto read_frags = [&](uint32_t st, int j, Frags& f) {
    const int q = PK ? 2 * j + g : 4 * g + j;
#pragma unroll
    for (int mb = 0; mb < G::MBW; ++mb) {
      const int r = (wm * G::MBW + mb) * 32 + c32;
      const uint32_t rowa = st + (uint32_t)(r * G::RB);
#pragma unroll
      for (int part = 0; part < PARTS; ++part)
        f.a[mb][part] = lds_read16(rowa + (uint32_t)(((PARTS * q + part) ^ (r % NPC)) * 16));
    }
#pragma unroll
    for (int nb = 0; nb < G::NBW; ++nb) {
      if (PK) {
        const int blk = wn * G::NBW + nb;
        f.w[nb] = lds_read16(st + G::ASTAGE + (uint32_t)((blk * 4 + j) * 1024 + lane * 16));
      } else {
        const int t = (wn * G::NBW + nb) * 32 + c32;
        f.w[nb] = lds_read16(st + G::ASTAGE + (uint32_t)(t * 128 + ((q ^ ((t >> 1) & 7)) * 16)));
      }
    }
  };
  auto fence = [&](Frags& f) {
#pragma unroll
    for (int mb = 0; mb < G::MBW; ++mb)
#pragma unroll
      for (int part = 0; part < PARTS; ++part) lds_fence_value(f.a[mb][part]);
#pragma unroll
    for (int nb = 0; nb < G::NBW; ++nb) lds_fence_value(f.w[nb]);
  };
  // split format: hi parts for every accumulator, then lo parts
  auto mfma_step = [&](const Frags& f) {
#pragma unroll
    for (int part = 0; part < PARTS; ++part)
#pragma unroll
      for (int mb = 0; mb < G::MBW; ++mb) {
#pragma unroll
        for (int nb = 0; nb < G::NBW; ++nb) {
          if (A16)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, f.a[mb][part]),
                                                                 __builtin_bit_cast(f16x8_t, f.w[nb]), acc[mb][nb], 0, 0, 0);
          else
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, f.a[mb][part]),
                                                                  __builtin_bit_cast(bf16x8_t, f.w[nb]), acc[mb][nb], 0, 0, 0);
        }
      }
  };

#pragma unroll
  for (int s = 0; s < G::NS - 1; ++s) issue(s);
  for (int it = 0; it < nloc; ++it) {
    wait_vmcnt<G::WAIT>();          // this wave's loads of chunk it have landed
    lds_wait();                     // and its reads of chunk it - 1 are done
    __builtin_amdgcn_s_barrier();   // ... in every wave: chunk it is complete, stage it - 1 is free
    issue(it + G::NS - 1);
    const uint32_t st = ring_addr + (uint32_t)((it % G::NS) * G::STAGE);
    Frags f0, f1;
    read_frags(st, 0, f0);
    lds_wait();
    fence(f0);
    read_frags(st, 1, f1);          // next k-step in flight during this one
    mfma_step(f0);
    lds_wait();
    fence(f1);
    read_frags(st, 2, f0);
    mfma_step(f1);
    lds_wait();
    fence(f0);
    read_frags(st, 3, f1);
    mfma_step(f0);
    lds_wait();
    fence(f1);
    mfma_step(f1);
  }

  // epilogue: element i of lane l is row 8 (i / 4) + 4 g + i % 4, column c32
#pragma unroll
  for (int mb = 0; mb < G::MBW; ++mb) {
#pragma unroll
    for (int nb = 0; nb < G::NBW; ++nb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int m = m0 + (wm * G::MBW + mb) * 32 + 8 * (i >> 2) + 4 * g + (i & 3);
        const float v = acc[mb][nb][i];
        if (EPI == EPI_SWIGLU) {
          // columns 0..15 of the block are gate values, 16..31 the matching up values
          const float up = __shfl_xor(v, 16, 64);
          const int j = blockIdx.x * G::OUT_COLS + 16 * (wn * G::NBW + nb) + (c32 & 15);
          if (m < M && c32 < 16 && j < N) {
            if (A16) reinterpret_cast<uint16_t*>(out)[(size_t)m * ldo + j] = f2h(silu(v) * up);
            else split_store(reinterpret_cast<bf16_t*>(out) + (size_t)m * 2 * ldo, j, silu(v) * up);
          }
        } else {
          const int n = blockIdx.x * G::BN + (wn * G::NBW + nb) * 32 + c32;
          if (m < M && n < N) out[blockIdx.z * split_stride + (size_t)m * ldo + n] = v;
        }
      }
    }
  }
}

// ---------------------------------------------------------------- VALU path
template <typename WT, bool SPLIT, int EPI>
__global__ __launch_bounds__(256) void gemm_valu_kernel(
    const void* __restrict__ Av, const WT* __restrict__ W, int M, int N, int K, int kper,
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
      float a = 0.f;
      if (m < M && k < ke) {
        if (SPLIT) a = split_load(reinterpret_cast<const bf16_t*>(Av) + (size_t)m * 2 * K, k);
        else a = reinterpret_cast<const float*>(Av)[(size_t)m * K + k];
      }
      As[r][c] = a;
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
        act_store<SPLIT>(out, m, ldo, n, silu(acc[0][i][jj]) * acc[NW - 1][i][jj]);
      else
        out[blockIdx.z * split_stride + (size_t)m * ldo + n] = acc[0][i][jj];
    }
}

template <int BMT, int BNT, int NST, int EPI, bool PK = false, bool A16 = false>
hipError_t run_mfma(const GemmArgs& a, int S, int cps, hipStream_t st) {
  constexpr int NW = (BMT >= 128) ? 8 : 4;    // 128-row and larger tiles: two waves per SIMD
  using G = GemmShape<BMT, BNT, NST, NW, A16>;
  const int cols = (EPI == EPI_SWIGLU) ? G::OUT_COLS : G::BN;
  dim3 grid((a.N + cols - 1) / cols, (a.M + BMT - 1) / BMT, S);
  hipLaunchKernelGGL((gemm_mfma_kernel<BMT, BNT, NST, EPI, NW, PK, A16>), grid, dim3(64 * NW), 0, st,
                     (const bf16_t*)a.A, (const bf16_t*)(PK ? a.Wp : a.W), a.M, a.N, a.K, cps, a.out, a.ldo,
                     a.split_stride);
  return hipGetLastError();
}

template <int EPI>
hipError_t dispatch_mfma(const GemmArgs& a, int S, int cps, hipStream_t st) {
  if (a.Wp && a.M > 64) {
    // Per MFMA a wave of a 128 x 128 tile reads 1.25 KB of fragments from LDS
    // (fp16: 1 activation + 4 weight fragments for 4 MFMAs), more than the LDS
    // delivers at the matrix cores' rate.  A 256 x 256 fp16 tile (2 + 4
    // fragments for 8 MFMAs) and a 128 x 256 split tile (hi and lo: 2 + 4 for
    // 8) need 0.75 KB, but their grids fill the 256 CUs only for large M x N.
    const int rows = EPI == EPI_SWIGLU ? 2 * a.N : a.N;
    auto tiles = [&](int bm, int bn) { return (long)((a.M + bm - 1) / bm) * ((rows + bn - 1) / bn) * S; };
    if (a.a16)
      return tiles(256, 256) >= 128 ? run_mfma<256, 256, 2, EPI, true, true>(a, S, cps, st)
                                    : run_mfma<128, 128, 3, EPI, true, true>(a, S, cps, st);
    return tiles(128, 256) >= 256 ? run_mfma<128, 256, 2, EPI, true, false>(a, S, cps, st)
                                  : run_mfma<128, 128, 3, EPI, true, false>(a, S, cps, st);
  }
  if (a.M <= 32) return run_mfma<32, 128, 4, EPI>(a, S, cps, st);
  if (a.M <= 64) return run_mfma<64, 128, 4, EPI>(a, S, cps, st);
  return run_mfma<128, 128, 3, EPI>(a, S, cps, st);
}

template <typename WT, bool SPLIT>
hipError_t run_valu(const GemmArgs& a, int S, int kper, hipStream_t st) {
  dim3 grid((a.N + 31) / 32, (a.M + 31) / 32, S);
  if (a.epi == EPI_SWIGLU)
    hipLaunchKernelGGL((gemm_valu_kernel<WT, SPLIT, EPI_SWIGLU>), grid, dim3(256), 0, st, a.A,
                       (const WT*)a.W, a.M, a.N, a.K, kper, a.out, a.ldo, a.split_stride);
  else
    hipLaunchKernelGGL((gemm_valu_kernel<WT, SPLIT, EPI_PARTIAL>), grid, dim3(256), 0, st, a.A,
                       (const WT*)a.W, a.M, a.N, a.K, kper, a.out, a.ldo, a.split_stride);
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
  // packed weights take 128-row tiles (M > 64); fp16 activations need them
  if ((a.a16 && (!a.Wp || a.M <= 64)) || (a.Wp && (!mfma || (a.epi == EPI_SWIGLU && a.N % 16))))
    return hipErrorInvalidValue;
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
  if (a.dt == DT_BF16) return run_valu<bf16_t, true>(a, S, kper, st);
  return run_valu<float, false>(a, S, kper, st);
}

}  // namespace tandem
