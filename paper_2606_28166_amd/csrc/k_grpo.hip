// k_grpo.hip — the senior-only GRPO loss pieces over a batch of tandem
// rollouts (section 3.4, the L_TRL equation; Algorithm 1's update half).
//
// Per rollout s = j G + i: the group-relative advantage of its binary reward,
// normalised by the sample standard deviation of the group's G rewards
// (+1e-6).  Per position t < length[s] that the senior emitted (owner != 0):
// rho = exp(logp_new - logp_old) and GRPO's clipped term
// min(rho A, clip(rho, 1 - eps, 1 + eps) A).  The loss is minus the mean of
// those terms over every masked position of the batch; its gradient with
// respect to logp_new is -rho A / N where the unclipped term is the minimum
// and 0 elsewhere (junior positions, positions past the length, clipped
// terms).
//
// Two launches, HBM-streaming over the [S][T] arenas: per-rollout advantage
// and masked count; per-(chunk, rollout) terms, gradient and a partial sum.
// The workgroup that counts itself last on a ticket sums the partials in
// double in a fixed order (index order, whoever is last), so the loss is
// deterministic.  Partials are exchanged through agent-scope stores and
// loads, which are coherent across the chips' separate L2 caches; the ticket
// is counted with release-acquire ordering at agent scope, so the last
// workgroup reads every partial after its store.
#include <mutex>

#include "common.h"
#include "kernels.h"

namespace tandem {
namespace {

constexpr int kGrpoNT = 256;

__device__ __forceinline__ void st_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ __launch_bounds__(kGrpoNT) void grpo_adv_kernel(GrpoArgs a) {
  __shared__ float red[kGrpoNT / kWave];
  const int s = blockIdx.x, tid = threadIdx.x;
  const int j0 = (s / a.G) * a.G;
  float sr = 0.f;
  for (int i = tid; i < a.G; i += kGrpoNT) sr += a.rewards[j0 + i];
  const float mean = block_sum<kGrpoNT>(sr, red) / (float)a.G;
  float sq = 0.f;
  for (int i = tid; i < a.G; i += kGrpoNT) {
    const float d = a.rewards[j0 + i] - mean;
    sq += d * d;
  }
  sq = block_sum<kGrpoNT>(sq, red);
  const float sd = a.G > 1 ? sqrtf(sq / (float)(a.G - 1)) : 0.f;
  const int len = min(max(a.length[s], 0), a.T);
  const uint8_t* own = a.owner + (size_t)s * a.T;
  float c = 0.f;                             // exact: a row holds < 2^24 positions
  for (int t = tid; t < len; t += kGrpoNT) c += own[t] != 0 ? 1.f : 0.f;
  c = block_sum<kGrpoNT>(c, red);
  if (tid == 0) {
    a.adv[s] = (a.rewards[s] - mean) / (sd + 1e-6f);
    a.cnt[s] = (int32_t)c;
    if (s == 0) __hip_atomic_store(a.ticket, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

__global__ __launch_bounds__(kGrpoNT) void grpo_loss_kernel(GrpoArgs a) {
  __shared__ float red[kGrpoNT / kWave];
  const int chunk = blockIdx.x, s = blockIdx.y, tid = threadIdx.x;
  float n = 0.f;                             // exact: the batch holds < 2^24 positions
  for (int i = tid; i < a.S; i += kGrpoNT) n += (float)a.cnt[i];
  n = block_sum<kGrpoNT>(n, red);
  const float A = a.adv[s];
  const float lo_c = 1.f - a.eps, hi_c = 1.f + a.eps;
  const float inv_n = n > 0.f ? 1.f / n : 0.f;
  const int len = min(max(a.length[s], 0), a.T);
  const size_t row = (size_t)s * a.T;
  float acc = 0.f;
#pragma unroll
  for (int k = 0; k < kGrpoChunk / kGrpoNT; ++k) {
    const int t = chunk * kGrpoChunk + k * kGrpoNT + tid;
    if (t >= a.T) break;
    float g = 0.f;
    if (t < len && a.owner[row + t] != 0) {
      const float lo = a.logp_old[row + t];
      const float ln = a.logp_new ? a.logp_new[row + t] : lo;
      const float rho = expf(ln - lo);
      const float un = rho * A;
      const float cl = fminf(fmaxf(rho, lo_c), hi_c) * A;
      acc += fminf(un, cl);
      g = un <= cl ? -un * inv_n : 0.f;
    }
    if (a.grad) a.grad[row + t] = g;
  }
  acc = block_sum<kGrpoNT>(acc, red);
  const int np = a.S * a.n_chunks;
  __shared__ int last;
  if (tid == 0) {
    st_dev(a.part + (size_t)s * a.n_chunks + chunk, acc);
    // release: the partial is visible before the count; acquire: the last
    // one to count sees every other workgroup's partial
    last = __hip_atomic_fetch_add(a.ticket, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT) == np - 1;
  }
  __syncthreads();
  if (!last) return;
  // the last workgroup: every partial has been stored; the fence orders this
  // workgroup's loads after the acquire of its first thread
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  __shared__ double dred[kGrpoNT];
  double sum = 0.0;
  for (int i = tid; i < np; i += kGrpoNT) sum += (double)ld_dev(a.part + i);
  dred[tid] = sum;
  __syncthreads();
  for (int w = kGrpoNT / 2; w > 0; w >>= 1) {
    if (tid < w) dred[tid] += dred[tid + w];
    __syncthreads();
  }
  if (tid == 0) {
    a.loss[0] = n > 0.f ? (float)(-dred[0] / (double)n) : 0.f;
    a.n_masked[0] = (int32_t)n;
    __hip_atomic_store(a.ticket, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// The allocation-free entry point's workspace: one array per device, kept
// until the process ends.  Host code uses its device address from
// hipGetSymbolAddress (taken once per device), never the array's name.
static __device__ __align__(256) unsigned char scratch[kGrpoStaticBytes];

}  // namespace

hipError_t grpo_static_workspace(void** ptr) {
  static std::mutex mu;
  static void* addr[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

hipError_t launch_grpo(const GrpoArgs& a, hipStream_t st) {
  grpo_adv_kernel<<<a.S, kGrpoNT, 0, st>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  grpo_loss_kernel<<<dim3(a.n_chunks, a.S), kGrpoNT, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace tandem
