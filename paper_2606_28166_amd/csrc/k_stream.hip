// Decode projections: C = A . W^T for at most 128 activation rows, streaming
// the weights from HBM straight into registers.
//
// At decode a projection is a wide, skinny product: every weight is used by
// only the M <= 128 activation rows, so the kernel is a weight stream and its
// speed is the bytes it keeps in flight.  Two things make that stream fast on
// gfx950:
//   * The weights are packed once (pack_weights_kernel, at init) into MFMA
//     fragment order: a 32-row x 16-k block is one contiguous 1 KB fragment
//     whose 64 lanes each hold the 8 k-values one lane of
//     v_mfma_f32_32x32x16_bf16 consumes.  Every weight load is then one
//     coalesced 1 KB piece per wave, issued as a non-temporal buffer load
//     straight into VGPRs, NS - 1 chunks ahead of the arithmetic (512 KB of
//     register file per compute unit holds far more bytes in flight than the
//     160 KB of LDS).
//   * The activations are the operand every wave shares; they stream
//     through an NS-stage LDS ring by direct global->LDS loads, XOR-swizzled
//     so the fragment reads are free of bank conflicts.  They come in one of
//     two formats: split (bf16 high and low parts, two MFMAs per fragment,
//     fp32-level inputs: QKV and O, whose results feed the attention) or
//     fp16 (one MFMA per fragment against an fp16 copy of the weights: the
//     FFN and the LM head).  Every activation byte delivered to the CU is
//     traffic beside the weight stream: at 128 rows the split tile is twice
//     the bytes of its weights, the fp16 tile as many, which is most of the
//     difference in speed between the two.
// A workgroup is 4 waves, one per SIMD.  Wave w owns 32-row weight block w
// of the item and all MB 32-row activation blocks.  The work is a list of
// items (a group of 128 weight rows x one K slice); the grid is at most one
// workgroup per compute unit
// and each workgroup walks its items as one continuous chunk stream, so the
// prefetch runs on across item boundaries.  K slices > 1 write split-K
// partial tiles that the consuming kernel sums in a fixed order.
//
// MFMA operand layout (32x32x16): lane l supplies row / column l % 32 and
// the 8 k-values 8 (l / 32) .. +7 of the 16-value k-step; result element i
// of lane l is row 8 (i / 4) + 4 (l / 32) + i % 4, column l % 32.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace tandem {

namespace {

constexpr int SBK = 64;            // k-values per chunk (4 k-steps of 16)
constexpr int SNW = 4;             // waves per workgroup

// pair_rows F > 0 (a [2F][K] gate/up matrix): packed block b holds gate rows
// 16 b .. 16 b + 15 in its first 16 rows and the matching up rows F + 16 b ..
// in its last 16, so one MFMA output tile holds both halves of 16 SwiGLU
// outputs.
__global__ __launch_bounds__(256) void pack_weights_kernel(const bf16_t* __restrict__ W, int N, int K, int pair_rows,
                                                           int to_f16, bf16_t* __restrict__ out, long n_pieces) {
  const int ksn = K / 16;
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n_pieces; i += (long)gridDim.x * blockDim.x) {
    const long f = i >> 6;                        // fragment = (32-row block, 16-k step)
    const int lane = (int)(i & 63);
    const long nb = f / ksn;
    const int ks = (int)(f % ksn);
    const int c = lane & 31;
    const long row = pair_rows > 0 ? (c < 16 ? nb * 16 + c : pair_rows + nb * 16 + (c - 16)) : nb * 32 + c;
    const int k = 16 * ks + 8 * (lane >> 5);
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (row < N) v = *reinterpret_cast<const uint4*>(W + row * (long)K + k);
    if (to_f16) {
      uint32_t* w = reinterpret_cast<uint32_t*>(&v);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint16_t lo = __builtin_bit_cast(uint16_t, (_Float16)bf2f((bf16_t)(w[e] & 0xFFFFu)));
        const uint16_t hi = __builtin_bit_cast(uint16_t, (_Float16)bf2f((bf16_t)(w[e] >> 16)));
        w[e] = (uint32_t)lo | ((uint32_t)hi << 16);
      }
    }
    reinterpret_cast<uint4*>(out)[i] = v;
  }
}

// Both operands are loaded NS - 1 chunks ahead of the arithmetic: weights
// (from HBM) into a ring of NS register sets, activations (L2-resident) into
// an NS-stage LDS ring.  Iteration c issues A(c + NS - 1) then W(c + NS - 1).
// Vector loads retire in order, so the two rings must be equally deep: a
// wait for an activation stage also waits for every weight load issued
// before it.
template <int MB, int NS, bool A16>
struct StreamShape {
  static constexpr int BM = 32 * MB;                 // activation rows of the tile
  static constexpr int PARTS = A16 ? 1 : 2;          // MFMA operand parts per value (fp16, or bf16 hi + lo)
  static constexpr int RB = SBK * 2 * PARTS;         // bytes of one activation row per chunk
  static constexpr int NPC = RB / 16;                // 16-byte pieces per row (XOR-swizzled)
  static constexpr int RPI = 64 / NPC;               // rows per 1 KB DMA instruction
  static constexpr int ASTAGE = BM * RB;             // bytes of one activation stage
  static constexpr int NA = BM / (RPI * SNW);        // activation DMA instructions per wave per chunk
  static constexpr int NWL = 4;                      // weight loads per wave per chunk
  static constexpr int DW = NS - 1;                  // chunks in flight ahead of the arithmetic
  static constexpr int WAIT = (DW - 1) * (NA + NWL); // vmcnt once A(c) and W(c) have landed
  static_assert(NS >= 2, "ring of register sets and LDS stages");
  static_assert(NS * ASTAGE <= 160 * 1024, "LDS ring");
  static_assert(WAIT < 64, "vmcnt range");
  static_assert(NA >= 1, "at least one activation DMA per wave");
};

// Position in a workgroup's chunk stream: item (weight group x K slice) and
// chunk inside the item's K slice.  Uniform across the workgroup.
struct Cursor {
  int item, grp, s, c, nloc;
};

__device__ __forceinline__ float silu_f(float x) { return x / (1.f + expf(-x)); }

template <int MB, int NS, bool A16, int EPI>
__global__ __launch_bounds__(256) void gemm_stream_kernel(
    const bf16_t* __restrict__ A, const bf16_t* __restrict__ Wp, int M, int N, int K, int n_groups, int S, int cps,
    float* __restrict__ out, int ldo, long split_stride, SampleEpiArgs smp) {
  using G = StreamShape<MB, NS, A16>;
  constexpr int PARTS = G::PARTS, NPC = G::NPC;
  __shared__ __attribute__((aligned(1024))) unsigned char ring[NS * G::ASTAGE];
  // EPI_SAMPLE: an item's output tile (BM rows x 128 vocabulary entries,
  // padded rows) on its way from the MFMA layout to one row per thread pair
  constexpr int TSTR = 128 + 4;
  __shared__ __attribute__((aligned(16))) float tile[EPI == EPI_SAMPLE ? G::BM * TSTR : 1];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, c32 = lane & 31;
  const int nch = K / SBK;
  const int n_items = n_groups * S;
  const int nblk = (N + 31) >> 5;
  const int grid = gridDim.x;
  if ((int)blockIdx.x >= n_items) return;

  auto set_item = [&](Cursor& u, int item) {
    u.item = item;
    u.s = item / n_groups;
    u.grp = item - u.s * n_groups;
    u.c = 0;
    u.nloc = min(cps, nch - u.s * cps);
  };
  // the load cursor stays on the last chunk once the stream is exhausted
  // (re-issuing it is a cache hit and keeps the wait counts uniform)
  auto advance = [&](Cursor& u) {
    if (u.c + 1 < u.nloc) { ++u.c; return; }
    if (u.item + grid < n_items) set_item(u, u.item + grid);
  };

  // Activation DMA: instruction i of wave w covers tile rows
  // r0 + RPI SNW i .. +RPI - 1 (r0 = RPI w + lane / NPC; a row is NPC 16-byte
  // pieces: split format 8 hi and 8 lo pieces, fp16 8 pieces); physical piece
  // lane % NPC holds logical piece (lane % NPC) ^ (row % NPC).
  const int r0 = G::RPI * wave + lane / NPC;
  const int lc = (lane % NPC) ^ (r0 % NPC);
  const size_t lda = (size_t)K * PARTS;                    // row stride (2-byte elements)
  const __amdgpu_buffer_rsrc_t wr = buf_rsrc(Wp, (uint32_t)((size_t)nblk * (K / 16) * 1024));
  const int kfr = K / 16;                                  // fragments per 32-row block

  u32x4_t wb[NS][4];
  auto issue_a = [&](const Cursor& u, int stage) {
    const int kc = u.s * cps + u.c;
    unsigned char* st = ring + stage * G::ASTAGE;
#pragma unroll
    for (int i = 0; i < G::NA; ++i) {
      const bf16_t* src = A + (size_t)min(r0 + G::RPI * SNW * i, M - 1) * lda + (size_t)kc * PARTS * SBK + lc * 8;
      load_lds16(src, st + 4 * (SNW * i + wave) * 256);
    }
  };
  auto issue_w = [&](const Cursor& u, u32x4_t (&w)[4]) {
    const int kc = u.s * cps + u.c;
    const int nb = min(u.grp * SNW + wave, nblk - 1);
    const int base = (nb * kfr + 4 * kc) * 1024 + lane * 16;
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = buf_load16_nt(wr, base + j * 1024, 0);
  };
  // keeps the loads issued so far above the arithmetic of this chunk and
  // makes the compiler wait for this chunk's weights here, not earlier
  auto pin = [&](u32x4_t (&w)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) asm volatile("" : "+v"(w[j]) : : "memory");
  };

  f32x16_t acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x16_t{};

  const uint32_t ring_addr = lds_addr_of(ring);
  // A fragments of k-step j (k-values 16 j + 8 g .. +7 of the chunk = group 2 j + g:
  // pieces 2 q and 2 q + 1 of a split row, piece q of an fp16 row)
  auto read_a = [&](uint32_t st, int j, u32x4_t (&f)[MB][PARTS]) {
    const int q = 2 * j + g;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int r = mb * 32 + c32;
      const uint32_t row = st + (uint32_t)(r * G::RB);
#pragma unroll
      for (int part = 0; part < PARTS; ++part)
        f[mb][part] = lds_read16(row + (uint32_t)(((PARTS * q + part) ^ (r % NPC)) * 16));
    }
  };
  auto fence_a = [&](u32x4_t (&f)[MB][PARTS]) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int part = 0; part < PARTS; ++part) lds_fence_value(f[mb][part]);
  };
  // one chunk = 4 k-steps; the A fragments of k-step j + 1 are read while the
  // MFMAs of k-step j run (split format: high parts of every block, then low
  // parts, so consecutive MFMAs never share an accumulator when MB > 1)
  auto compute = [&](int stage, u32x4_t (&w)[4]) {
    const uint32_t st = ring_addr + (uint32_t)(stage * G::ASTAGE);
    u32x4_t fa[MB][PARTS], fb[MB][PARTS];
    read_a(st, 0, fa);
    pin(w);
    lds_wait();
    fence_a(fa);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      u32x4_t (&cur)[MB][PARTS] = (j & 1) ? fb : fa;
      u32x4_t (&nxt)[MB][PARTS] = (j & 1) ? fa : fb;
      if (j < 3) read_a(st, j + 1, nxt);
#pragma unroll
      for (int part = 0; part < PARTS; ++part)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          if (A16)
            acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, cur[mb][part]),
                                                             __builtin_bit_cast(f16x8_t, w[j]), acc[mb], 0, 0, 0);
          else
            acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, cur[mb][part]),
                                                              __builtin_bit_cast(bf16x8_t, w[j]), acc[mb], 0, 0, 0);
        }
      if (j < 3) {
        lds_wait();
        fence_a(nxt);
      }
    }
  };
  // EPI_SAMPLE running state of row ts_m over columns 64 ts_h .. + 63 of
  // every item this workgroup takes: log-sum-exp of the scores (senior head)
  // and the top two Gumbel-perturbed scores (rows this model owns)
  const int ts_m = tid >> 1, ts_h = tid & 1;
  float ts_ms = -INFINITY, ts_ls = 0.f;
  Top2 ts_top{-INFINITY, 0x7FFFFFFF, -INFINITY};
  bool ts_live = false, ts_own = false;
  if (EPI == EPI_SAMPLE && ts_m < M) {
    const int s = smp.act[ts_m];
    ts_live = smp.done[s] == 0;
    ts_own = (smp.owner[s] != 0 ? 1 : 0) == smp.model;
  }
  auto epilogue = [&](const Cursor& u) {
    const int nb = u.grp * SNW + wave;                   // this wave's 32-row weight block
    if (EPI == EPI_SAMPLE) {
      const int v0 = u.grp * 128 + 64 * ts_h;
      const int lim = N - v0;                            // entries of this thread's half inside the vocabulary
      const bool sen = smp.model == 1, work = ts_live && (sen || ts_own);
      // the first half of this thread's noise, requested before the tile
      // goes through LDS (the second half as the first is consumed)
      const float4* nrow = reinterpret_cast<const float4*>(smp.noise + (size_t)ts_m * N + v0);
      auto noise4 = [&](int q) { return 4 * q < lim ? nrow[q] : make_float4(0.f, 0.f, 0.f, 0.f); };
      float4 gn[8];
      if (work && ts_own) {
#pragma unroll
        for (int q = 0; q < 8; ++q) gn[q] = noise4(q);
      }
      // scores s = (z + b 1[v = eos]) / T into the tile
      const float inv_t = 1.f / smp.temp;
      const float eb = u.grp * 128 + wave * 32 + c32 == smp.eos_id ? smp.eos_bias * inv_t : 0.f;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int m = mb * 32 + 8 * (i >> 2) + 4 * g + (i & 3);
          tile[m * TSTR + wave * 32 + c32] = fmaf(acc[mb][i], inv_t, eb);
          acc[mb][i] = 0.f;
        }
      __syncthreads();
      if (work) {
        // the four scores of quad q of this half (-inf past the vocabulary),
        // read from the tile on every pass instead of held in registers
        const float4* trow = reinterpret_cast<const float4*>(tile + ts_m * TSTR + 64 * ts_h);
        auto quad = [&](int q, float* sc) {
          const float4 z = trow[q];
          sc[0] = 4 * q < lim ? z.x : -INFINITY;
          sc[1] = 4 * q + 1 < lim ? z.y : -INFINITY;
          sc[2] = 4 * q + 2 < lim ? z.z : -INFINITY;
          sc[3] = 4 * q + 3 < lim ? z.w : -INFINITY;
        };
        if (sen) {
          // log-sum-exp of the 64 scores, folded into the running pair
          float mx = -INFINITY;
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            float sc[4];
            quad(q, sc);
            mx = fmaxf(fmaxf(mx, fmaxf(sc[0], sc[1])), fmaxf(sc[2], sc[3]));
          }
          if (mx > -INFINITY) {
            const float off = -mx * 1.4426950408889634f;
            float l0 = 0.f, l1 = 0.f;
#pragma unroll
            for (int q = 0; q < 16; ++q) {
              float sc[4];
              quad(q, sc);
              l0 += __builtin_amdgcn_exp2f(fmaf(sc[0], 1.4426950408889634f, off));
              l1 += __builtin_amdgcn_exp2f(fmaf(sc[1], 1.4426950408889634f, off));
              l0 += __builtin_amdgcn_exp2f(fmaf(sc[2], 1.4426950408889634f, off));
              l1 += __builtin_amdgcn_exp2f(fmaf(sc[3], 1.4426950408889634f, off));
            }
            merge_lse(ts_ms, ts_ls, mx, l0 + l1);
          }
        }
        if (ts_own) {
          // top two of s + noise (ties to the smaller index), then into the running state
          float b = -INFINITY, s2 = -INFINITY;
          int bi = 0x7FFFFFFF;
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            const float gv[4] = {gn[q & 7].x, gn[q & 7].y, gn[q & 7].z, gn[q & 7].w};
            if (q < 8) gn[q] = noise4(q + 8);
            float sc[4];
            quad(q, sc);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float val = sc[e] + gv[e];
              const bool up = val > b;
              s2 = up ? b : fmaxf(s2, val);
              bi = up ? v0 + 4 * q + e : bi;
              b = up ? val : b;
            }
          }
          ts_top = merge_top2(ts_top, Top2{b, bi, s2});
        }
      }
      __syncthreads();                                   // the tile is written again by the next item
      return;
    }
    if (EPI == EPI_SWIGLU) {
      // columns c < 16 of a block are gate sums, c + 16 the matching up sums
      // (pair-interleaved packing); output column 16 nb + c, in the input's
      // format (fp16, or split)
      const int j = nb * 16 + (c32 & 15);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float v = acc[mb][i];
          const float up = __shfl_xor(v, 16, 64);
          const int m = mb * 32 + 8 * (i >> 2) + 4 * g + (i & 3);
          if (m < M && c32 < 16 && j < ldo) {
            if (A16) reinterpret_cast<uint16_t*>(out)[(size_t)m * ldo + j] = f2h(silu_f(v) * up);
            else split_store(reinterpret_cast<bf16_t*>(out) + (size_t)m * 2 * ldo, j, silu_f(v) * up);
          }
          acc[mb][i] = 0.f;
        }
      return;
    }
    float* o = out + (size_t)u.s * split_stride;
    const int n = nb * 32 + c32;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int m = mb * 32 + 8 * (i >> 2) + 4 * g + (i & 3);
        if (m < M && n < N) o[(size_t)m * ldo + n] = acc[mb][i];
        acc[mb][i] = 0.f;
      }
  };

  // Every item's chunk count is a multiple of NS (the host guarantees
  // K % (64 NS) == 0 and cps % NS == 0), so chunk c of an item sits in
  // register set and LDS stage c % NS: compile-time indices below.
  Cursor la, cp;                        // load cursor (both operands), compute cursor
  set_item(la, blockIdx.x);
#pragma unroll
  for (int d = 0; d < G::DW; ++d) {
    issue_a(la, d);
    issue_w(la, wb[d]);
    advance(la);
  }
  for (int item = blockIdx.x; item < n_items; item += grid) {
    set_item(cp, item);
    for (int c0 = 0; c0 < cp.nloc; c0 += NS) {
#pragma unroll
      for (int u = 0; u < NS; ++u) {
        wait_vmcnt<G::WAIT>();          // A(c) and W(c) of this wave have landed
        lds_wait();                     // and its LDS reads of the previous chunk are done
        __builtin_amdgcn_s_barrier();   // ... in every wave: A(c) is complete, stage c - 1 is free
        issue_a(la, (u + G::DW) % NS);
        issue_w(la, wb[(u + G::DW) % NS]);
        advance(la);
        compute(u, wb[u]);
      }
    }
    epilogue(cp);
  }
  if (EPI == EPI_SAMPLE) {
    // the two halves of each row, then one partial per (row, workgroup)
    const float m2 = __shfl_xor(ts_ms, 1, 64), l2 = __shfl_xor(ts_ls, 1, 64);
    merge_lse(ts_ms, ts_ls, m2, l2);
    const Top2 B{__shfl_xor(ts_top.b, 1, 64), __shfl_xor(ts_top.i, 1, 64), __shfl_xor(ts_top.s, 1, 64)};
    ts_top = merge_top2(ts_top, B);
    if (ts_h == 0 && ts_m < M) {
      float* p = smp.part + ((size_t)ts_m * smp.n_part + blockIdx.x) * 5;
      p[0] = ts_ms; p[1] = ts_ls; p[2] = ts_top.b; p[3] = __int_as_float(ts_top.i); p[4] = ts_top.s;
    }
  }
}

template <int MB, bool A16, int EPI>
hipError_t run_stream(const GemmStreamArgs& a, int grid, hipStream_t st) {
  constexpr int NS = kStreamStages;
  hipLaunchKernelGGL((gemm_stream_kernel<MB, NS, A16, EPI>), dim3(grid), dim3(64 * SNW), 0, st,
                     (const bf16_t*)a.A, (const bf16_t*)a.Wp, a.M, a.N, a.K, a.n_groups, a.S, a.cps, a.out, a.ldo,
                     a.split_stride, a.smp);
  return hipGetLastError();
}

template <int MB>
hipError_t dispatch_epi(const GemmStreamArgs& a, int grid, hipStream_t st) {
  if (a.a16 && a.epi == EPI_SAMPLE) return run_stream<MB, true, EPI_SAMPLE>(a, grid, st);
  if (a.a16)
    return a.epi == EPI_SWIGLU ? run_stream<MB, true, EPI_SWIGLU>(a, grid, st)
                               : run_stream<MB, true, EPI_PARTIAL>(a, grid, st);
  return a.epi == EPI_SWIGLU ? run_stream<MB, false, EPI_SWIGLU>(a, grid, st)
                             : run_stream<MB, false, EPI_PARTIAL>(a, grid, st);
}

}  // namespace

size_t packed_weight_bytes(int N, int K) { return (size_t)((N + 31) / 32) * 32 * (size_t)K * 2; }

bool stream_gemm_ok(int M, int N, int K) {
  return M >= 1 && M <= kStreamMaxRows && K % (SBK * kStreamStages) == 0 && N >= 1 &&
         packed_weight_bytes(N, K) < ((size_t)1 << 31);
}

hipError_t launch_pack_weights(const void* W, int N, int K, int pair_rows, bool to_f16, void* out, hipStream_t st) {
  if (pair_rows > 0 && (N != 2 * pair_rows || pair_rows % 16)) return hipErrorInvalidValue;
  const long pieces = (long)((N + 31) / 32) * (K / 16) * 64;
  const long blocks = std::min<long>((pieces + 255) / 256, 65536);
  hipLaunchKernelGGL(pack_weights_kernel, dim3((unsigned)blocks), dim3(256), 0, st, (const bf16_t*)W, N, K, pair_rows,
                     to_f16 ? 1 : 0, (bf16_t*)out, pieces);
  return hipGetLastError();
}

StreamPlan plan_stream_gemm(int M, int N, int K, int n_cu, size_t ws_floats, int mode) {
  // Cost in chunk times of the busiest workgroup: items are dealt round-robin
  // to at most n_cu workgroups, each item costs its chunks plus about two for
  // its epilogue and pipeline refill; K slices > 1 also pay for the partial
  // tiles the consumer reads back (in 32 KB-per-unit chunks spread over the
  // device) and, for SwiGLU, for the separate pass that applies it.
  const int nch = K / SBK;
  const int groups = (N + 127) / 128;
  const int smax = mode == kPlanStore ? 1 : std::min(kSplitMaxStream, nch / kStreamStages);
  double best = 1e300;
  StreamPlan pl{1, 1, nch, groups, std::min(groups, n_cu)};
  for (int S = 1; S <= std::max(1, smax); ++S) {
    const int cps = ((nch + S - 1) / S + kStreamStages - 1) / kStreamStages * kStreamStages;
    const int su = (nch + cps - 1) / cps;
    if (su != S) continue;
    if (S > 1 && (size_t)S * M * N > ws_floats) break;
    const long items = (long)groups * S;
    double cost = (double)((items + n_cu - 1) / n_cu) * (cps + 2);
    if (S > 1) {
      cost += (double)S * M * N * 4 / ((double)n_cu * 32768);
      if (mode == kPlanSwiglu) cost += 4 + (double)S * M * N * 4 / ((double)n_cu * 16384);
    }
    if (cost < best) {
      best = cost;
      pl = StreamPlan{1, S, cps, groups, (int)std::min<long>(items, n_cu)};
    }
  }
  return pl;
}

hipError_t launch_gemm_stream(const GemmStreamArgs& a, hipStream_t st) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (!stream_gemm_ok(a.M, a.N, a.K) || a.S < 1 || a.cps < 1 || a.n_groups < 1 || a.nbw != 1 ||
      a.cps % kStreamStages != 0 || (long)a.S * a.cps < a.K / SBK || (long)(a.S - 1) * a.cps >= a.K / SBK ||
      a.grid < 1)
    return hipErrorInvalidValue;
  if (a.epi == EPI_SWIGLU && (a.S != 1 || a.N % 32)) return hipErrorInvalidValue;
  if (a.epi == EPI_SAMPLE && (a.S != 1 || !a.a16 || a.N % 4 || !a.smp.noise || !a.smp.part || !a.smp.act ||
                              !a.smp.owner || !a.smp.done || a.smp.n_part < std::min(a.grid, a.n_groups)))
    return hipErrorInvalidValue;
  const int grid = std::min(a.grid, a.n_groups * a.S);
  if (a.M <= 32) return dispatch_epi<1>(a, grid, st);
  if (a.M <= 64) return dispatch_epi<2>(a, grid, st);
  return dispatch_epi<4>(a, grid, st);
}

}  // namespace tandem
