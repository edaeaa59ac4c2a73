// Device-side helpers shared by the gfx950 kernels of libtandem.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tandem {

typedef uint16_t bf16_t;   // bf16 bit pattern
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float((uint32_t)b << 16); }

// float -> bf16, round to nearest even (inputs are finite)
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ __forceinline__ static float load(const float* p) { return *p; }
  __device__ __forceinline__ static void store(float* p, float v) { *p = v; }
};
template <> struct Elem<bf16_t> {
  __device__ __forceinline__ static float load(const bf16_t* p) { return bf2f(*p); }
  __device__ __forceinline__ static void store(bf16_t* p, float v) { *p = f2bf(v); }
};

template <typename T> __device__ __forceinline__ float ld(const T* p) { return Elem<T>::load(p); }
template <typename T> __device__ __forceinline__ void st(T* p, float v) { Elem<T>::store(p, v); }

// ------------------------------------------------------------ split format
// Activations of bf16 models are stored "split": each group of 8 values is
// 16 bf16 words, the 8 high parts hi = bf16(x) followed by the 8 low parts
// lo = bf16(x - hi).  hi + lo carries x to about 2^-16 relative, in the
// 4 bytes per value of fp32, and both halves are ready-made MFMA operands.
__device__ __forceinline__ void split_store(bf16_t* row, int k, float x) {
  const bf16_t h = f2bf(x);
  bf16_t* p = row + (k >> 3) * 16 + (k & 7);
  p[0] = h;
  p[8] = f2bf(x - bf2f(h));
}
__device__ __forceinline__ float split_load(const bf16_t* row, int k) {
  const bf16_t* p = row + (k >> 3) * 16 + (k & 7);
  return bf2f(p[0]) + bf2f(p[8]);
}

// ------------------------------------------------------------ fp16 format
// The inputs of the FFN projections and the LM head at decode are plain
// fp16 (one rounding, 2^-11 relative; the two-part split is kept where the
// attention consumes the result): 2 bytes per value and one MFMA per
// fragment.  Values are saturated to the fp16 range.
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
__device__ __forceinline__ uint16_t f2h(float x) {
  return __builtin_bit_cast(uint16_t, (_Float16)fminf(fmaxf(x, -65504.f), 65504.f));
}

// Activation formats written by the norm passes.
enum { ACT_F32 = 0, ACT_SPLIT = 1, ACT_F16 = 2 };

// Activation row store in either format (split for bf16 models, plain fp32 otherwise).
template <bool SPLIT>
__device__ __forceinline__ void act_store(void* base, size_t row, int K, int k, float x) {
  if (SPLIT) split_store(reinterpret_cast<bf16_t*>(base) + row * 2 * (size_t)K, k, x);
  else reinterpret_cast<float*>(base)[row * (size_t)K + k] = x;
}

// s_waitcnt that waits only for vector memory operations: vmcnt <= n.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
__device__ __forceinline__ void wait_lgkm0() {
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
}

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

// 16 bytes per lane from global memory straight into LDS at lds_base + 16 * lane.
__device__ __forceinline__ void load_lds16(const void* gsrc, void* lds_base) {
  __builtin_amdgcn_global_load_lds((glb_void_t*)gsrc, (lds_void_t*)lds_base, 16, 0, 0);
}
// Same, for data read once (non-temporal: not kept in the caches).
__device__ __forceinline__ void load_lds16_nt(const void* gsrc, void* lds_base) {
  __builtin_amdgcn_global_load_lds((glb_void_t*)gsrc, (lds_void_t*)lds_base, 16, 0, 2);
}

// LDS read the compiler does not see as a memory access: it then cannot
// conflate it with pending LDS-DMA writes (which would make it drain every
// outstanding load).  The caller must wait with lds_wait() before using the
// result and must order ring reuse with its own barriers.
// Tiled K/V cache.  A (slot, kv head) plane holds ctx_stride positions in
// chunks of 16; inside a chunk the elements sit in the order the decode
// attention MFMAs consume them, so every 64-lane load of a chunk is one
// contiguous 1 KB piece (for 16-bit elements).
//   K: piece dc (dims 32dc .. 32dc+31), lane g*16 + c16 holds position c16,
//      dims 32dc + 8g .. +7.
//   V: piece j (dims 32j .. 32j+31), lane g*16 + c16 holds positions
//      4g .. 4g+3 of dim 32j + c16, then of dim 32j + 16 + c16.
// Both are element indices inside the plane; hd is a multiple of 32.
__device__ __forceinline__ int kv_k_index(int p, int d, int hd) {
  return (p >> 4) * 16 * hd + ((((d >> 5) * 64) + ((d >> 3) & 3) * 16 + (p & 15)) << 3) + (d & 7);
}
__device__ __forceinline__ int kv_v_index(int p, int d, int hd) {
  const int j = p & 15;
  return (p >> 4) * 16 * hd + ((((d >> 5) * 64) + (j >> 2) * 16 + (d & 15)) << 3) + (((d >> 4) & 1) << 2) + (j & 3);
}

// Raw buffer access: a uniform base and a byte size (reads at or past the
// size return zeros), per-lane 32-bit byte offsets, a uniform byte offset.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ u32x4_t buf_load16(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
}
// Streaming read (non-temporal: data read once, not kept in the caches).
__device__ __forceinline__ u32x4_t buf_load16_nt(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 2);
}
__device__ __forceinline__ u32x2_t buf_load8(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
}

__device__ __forceinline__ u32x4_t lds_read16(uint32_t lds_addr) {
  u32x4_t r;
  asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(lds_addr));
  return r;
}
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// Ties a value to the preceding lds_wait() so no use is scheduled before it.
__device__ __forceinline__ void lds_fence_value(u32x4_t& v) { asm volatile("" : "+v"(v)); }
__device__ __forceinline__ uint32_t lds_addr_of(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Block-wide sum for blockDim.x == NT (multiple of 64); all threads get the result.
template <int NT>
__device__ __forceinline__ float block_sum(float v, float* red /* >= NT/64 floats */) {
  v = wave_sum(v);
  const int w = threadIdx.x / kWave, l = threadIdx.x % kWave;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NT / kWave; ++i) s += red[i];
  return s;
}

// ---------------------------------------------------------------- Philox4x32-10
// Salmon, Moraes, Dror & Shaw, SC'11: 10 rounds of
//   (c0,c1,c2,c3) -> (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0))
// with the key bumped by the Weyl constants between rounds.
struct u32x4 { uint32_t x, y, z, w; };

__device__ __forceinline__ u32x4 philox4x32_10(u32x4 c, uint32_t k0, uint32_t k1) {
  const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += W0; k1 += W1; }
    const uint32_t hi0 = __umulhi(M0, c.x), lo0 = M0 * c.x;
    const uint32_t hi1 = __umulhi(M1, c.z), lo1 = M1 * c.z;
    c = u32x4{hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0};
  }
  return c;
}

// Uniform on 2^23 points strictly inside (0,1): (2*(x>>9)+1) * 2^-24, exact in fp32.
__device__ __forceinline__ float uniform_open(uint32_t x) {
  return (float)((x >> 9) * 2u + 1u) * 5.9604644775390625e-08f;
}

// Standard Gumbel noise -log(-log u).
__device__ __forceinline__ float gumbel(uint32_t x) {
  return -logf(-logf(uniform_open(x)));
}

// The same through the hardware log2 (v_log_f32, about 1 ulp): -ln(-ln u)
// with ln y = log2(y) * ln 2.  u >= 2^-24 keeps both arguments normal.
__device__ __forceinline__ float gumbel_fast(uint32_t x) {
  const float ln2 = 0.6931471805599453f;
  const float a = -__builtin_amdgcn_logf(uniform_open(x)) * ln2;    // -ln u > 0
  return -__builtin_amdgcn_logf(a) * ln2;
}

// e^x through the hardware exp2 (v_exp_f32); x <= 0 here.
__device__ __forceinline__ float fast_exp(float x) {
  return __builtin_amdgcn_exp2f(x * 1.4426950408889634f);
}

// --------------------------------------------------------------- sampling
// Best and second-best Gumbel-perturbed score of a vocabulary range: b at
// index i, s the runner-up (ties go to the smaller index).
struct Top2 {
  float b; int i; float s;
};
__device__ __forceinline__ bool beats(float vb, int ib, float va, int ia) {
  return vb > va || (vb == va && ib < ia);
}
__device__ __forceinline__ Top2 merge_top2(Top2 A, Top2 B) {
  Top2 out;
  if (beats(B.b, B.i, A.b, A.i)) {
    out.b = B.b; out.i = B.i; out.s = fmaxf(fmaxf(A.s, B.s), A.b);
  } else {
    out.b = A.b; out.i = A.i; out.s = fmaxf(fmaxf(A.s, B.s), B.b);
  }
  return out;
}
// Running (max m, sum l of e^(v - m)) pairs merged.
__device__ __forceinline__ void merge_lse(float& m, float& l, float m2, float l2) {
  const float M = fmaxf(m, m2);
  if (M == -INFINITY) { m = M; l = 0.f; return; }
  l = l * expf(m - M) + l2 * expf(m2 - M);
  m = M;
}

}  // namespace tandem
