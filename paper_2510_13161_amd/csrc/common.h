// Device-side helpers shared by the verification kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace msd {

constexpr int kWave = 64;
constexpr int kMaxSlots = 64;
constexpr int kMaxKappa = 32;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Block topology, passed by value to kernels (no device upload needed).
// anc[i] bit a = slot a is an ancestor of slot i or i itself.
struct Topo {
  uint64_t anc[kMaxSlots];
  int32_t depth[kMaxSlots];
  int32_t parent[kMaxSlots];
  int32_t n_slots;
  int32_t max_depth;
};

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Eight fp32 values as bf16 hi + lo parts (x ~= hi + lo to ~16 bits).
__device__ __forceinline__ void split_vals(const float (&v)[8], bf16x8& hi, bf16x8& lo) {
  u32x4 h, l;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    h[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
    l[i] = pack_bf16x2(v[2 * i] - bf_lo(h[i]), v[2 * i + 1] - bf_hi(h[i]));
  }
  hi = __builtin_bit_cast(bf16x8, h);
  lo = __builtin_bit_cast(bf16x8, l);
}
__device__ __forceinline__ bf16x8 round_vals(const float (&v)[8]) {
  u32x4 h;
#pragma unroll
  for (int i = 0; i < 4; ++i) h[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
  return __builtin_bit_cast(bf16x8, h);
}

// LDS-only workgroup barrier: waits for this wave's LDS traffic, not for its
// outstanding global loads (a full __syncthreads would drain those too); the
// empty asm statements keep the compiler from moving memory accesses across.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0), vmcnt/expcnt left open
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt for at most n outstanding vector-memory loads (expcnt and
// lgkmcnt not waited on)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt field is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// 16-byte loads. Weights are streamed once per pass: non-temporal.
__device__ __forceinline__ bf16x8 load_nt(const uint16_t* p) {
  u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return __builtin_bit_cast(bf16x8, v);
}
__device__ __forceinline__ bf16x8 load16(const uint16_t* p) {
  u32x4 v = *reinterpret_cast<const u32x4*>(p);
  return __builtin_bit_cast(bf16x8, v);
}
__device__ __forceinline__ bf16x8 zero_bf16x8() {
  u32x4 z = {0u, 0u, 0u, 0u};
  return __builtin_bit_cast(bf16x8, z);
}

// Eight consecutive fp32 values split into bf16 hi + lo parts (x ~= hi + lo to
// about 16 significant bits): activations stay fp32 and enter the MFMA as two
// bf16 operands against the exact bf16 weights.
__device__ __forceinline__ void load_split8(const float* p, bf16x8& hi, bf16x8& lo) {
  const u32x4 a = *reinterpret_cast<const u32x4*>(p);
  const u32x4 b = *reinterpret_cast<const u32x4*>(p + 4);
  const float v[8] = {__uint_as_float(a[0]), __uint_as_float(a[1]), __uint_as_float(a[2]),
                      __uint_as_float(a[3]), __uint_as_float(b[0]), __uint_as_float(b[1]),
                      __uint_as_float(b[2]), __uint_as_float(b[3])};
  u32x4 h, l;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint16_t h0 = f2bf(v[2 * i]), h1 = f2bf(v[2 * i + 1]);
    const uint16_t l0 = f2bf(v[2 * i] - bf2f(h0)), l1 = f2bf(v[2 * i + 1] - bf2f(h1));
    h[i] = (uint32_t)h0 | ((uint32_t)h1 << 16);
    l[i] = (uint32_t)l0 | ((uint32_t)l1 << 16);
  }
  hi = __builtin_bit_cast(bf16x8, h);
  lo = __builtin_bit_cast(bf16x8, l);
}
// Same split for a pre-normalised operand: v = (x - mu) * s * g (+ b).
__device__ __forceinline__ void load_norm_split8(const float* x, const uint16_t* g,
                                                 const uint16_t* bsh, float mu, float s,
                                                 bool split, bf16x8& hi, bf16x8& lo) {
  const u32x4 a = *reinterpret_cast<const u32x4*>(x);
  const u32x4 b = *reinterpret_cast<const u32x4*>(x + 4);
  const u32x4 gw = *reinterpret_cast<const u32x4*>(g);
  u32x4 bw = {0u, 0u, 0u, 0u};
  if (bsh) bw = *reinterpret_cast<const u32x4*>(bsh);
  const float xv[8] = {__uint_as_float(a[0]), __uint_as_float(a[1]), __uint_as_float(a[2]),
                       __uint_as_float(a[3]), __uint_as_float(b[0]), __uint_as_float(b[1]),
                       __uint_as_float(b[2]), __uint_as_float(b[3])};
  u32x4 h, l;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float g0 = __uint_as_float(gw[i] << 16), g1 = __uint_as_float(gw[i] & 0xFFFF0000u);
    const float b0 = __uint_as_float(bw[i] << 16), b1 = __uint_as_float(bw[i] & 0xFFFF0000u);
    const float v0 = (xv[2 * i] - mu) * s * g0 + b0;
    const float v1 = (xv[2 * i + 1] - mu) * s * g1 + b1;
    const uint16_t h0 = f2bf(v0), h1 = f2bf(v1);
    h[i] = (uint32_t)h0 | ((uint32_t)h1 << 16);
    l[i] = split ? pack_bf16x2(v0 - bf2f(h0), v1 - bf2f(h1)) : 0u;
  }
  hi = __builtin_bit_cast(bf16x8, h);
  lo = __builtin_bit_cast(bf16x8, l);
}

__device__ __forceinline__ bf16x8 load_round8(const float* p) {
  const u32x4 a = *reinterpret_cast<const u32x4*>(p);
  const u32x4 b = *reinterpret_cast<const u32x4*>(p + 4);
  u32x4 h;
  h[0] = pack_bf16x2(__uint_as_float(a[0]), __uint_as_float(a[1]));
  h[1] = pack_bf16x2(__uint_as_float(a[2]), __uint_as_float(a[3]));
  h[2] = pack_bf16x2(__uint_as_float(b[0]), __uint_as_float(b[1]));
  h[3] = pack_bf16x2(__uint_as_float(b[2]), __uint_as_float(b[3]));
  return __builtin_bit_cast(bf16x8, h);
}

// D = A * B + C on a 16x16 tile, K = 32, bf16 inputs, fp32 accumulate.
// Lane l: A row l%16, k 8*(l/16)..+8; B column l%16, same k;
// D rows 4*(l/16)+r (r = 0..3), column l%16.
__device__ __forceinline__ floatx4 mfma16x16x32(bf16x8 a, bf16x8 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Order-preserving map of fp32 onto uint32 (larger float -> larger key).
__device__ __forceinline__ uint32_t ordered_bits(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float from_ordered_bits(uint32_t k) {
  uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
  return __uint_as_float(u);
}
// Ranking key: larger logit first, then smaller id. 0 = no candidate.
__device__ __forceinline__ uint64_t rank_key(float v, int32_t id) {
  return ((uint64_t)ordered_bits(v) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)id);
}
__device__ __forceinline__ int32_t key_id(uint64_t k) {
  return (int32_t)(0xFFFFFFFFu - (uint32_t)(k & 0xFFFFFFFFull));
}
__device__ __forceinline__ float key_val(uint64_t k) { return from_ordered_bits((uint32_t)(k >> 32)); }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint64_t w = __shfl_xor(v, o);
    v = w > v ? w : v;
  }
  return v;
}

// Cross-workgroup hand-off inside one kernel (split-K partials, attention
// chunks). The payload is written and read with agent-scope atomic accesses,
// which the gfx950 memory model implements as L2-coherent (sc1) stores and
// loads; the writer drains its stores (s_waitcnt) before bumping the counter.
// No whole-L2 writeback or invalidate is needed, unlike a device-scope fence.
__device__ __forceinline__ void store_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_coherent(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// make this wave's LDS writes visible to its own later LDS reads
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// all of this wave's memory accesses complete; the compiler moves none across
__device__ __forceinline__ void drain_stores() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0);
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ int counter_add(int32_t* c, int v) {
  return __hip_atomic_fetch_add(c, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void counter_reset(int32_t* c) {
  __hip_atomic_store(c, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// 8-byte variants of the coherent hand-off accesses (two floats at a time).
__device__ __forceinline__ void store_coherent2(float* p, float a, float b) {
  const uint64_t v = (uint64_t)__float_as_uint(a) | ((uint64_t)__float_as_uint(b) << 32);
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 load_coherent2(const float* p) {
  const uint64_t v = __hip_atomic_load(reinterpret_cast<uint64_t*>(const_cast<float*>(p)),
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float((uint32_t)v), __uint_as_float((uint32_t)(v >> 32)));
}

// 16-byte variants: buffer loads and stores with the same L2-coherent (sc1)
// policy, through a resource that covers the hand-off region. A wave's
// 16-byte-per-lane access to a contiguous 1 KB then moves whole cache lines;
// the 8-byte accesses above write each line in two masked halves, which the
// memory side pays for several times over.
constexpr int kCoherentPolicy = 16;  // the SC1 cache-policy bit
__device__ __forceinline__ __amdgpu_buffer_rsrc_t coherent_region(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ void store_coherent4(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, floatx4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, byte_off, 0, kCoherentPolicy);
}
__device__ __forceinline__ floatx4 load_coherent4(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, kCoherentPolicy);
}

// z * sigmoid(z) with the hardware exponential and reciprocal
__device__ __forceinline__ float silu(float z) { return z * __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }

// Activation image: the split-bf16 MFMA operand form of an activation matrix
// [M][K] (M padded to 16 MT rows). Element order [K/32][MT][2][64][8]: k-step
// ks, row tile mt, part (0 = hi, 1 = lo), lane l = row 16 mt + l%16 and
// columns 32 ks + 8 (l/16) .. +8. One k-step of one row tile is 1 KB of hi and
// 1 KB of lo: exactly the B operand of one MFMA 16x16x32 per part. Rows past
// M are zero.
__device__ __forceinline__ size_t img_offset(int ks, int mt, int MT, int lane) {
  return ((size_t)(ks * MT + mt) * 2) * 512 + (size_t)lane * 8;
}
// Eight values as the hi and lo words of one image lane.
__device__ __forceinline__ void split8_words(const float (&v)[8], u32x4& h, u32x4& l) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    h[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
    l[i] = pack_bf16x2(v[2 * i] - bf_lo(h[i]), v[2 * i + 1] - bf_hi(h[i]));
  }
}

}  // namespace msd
