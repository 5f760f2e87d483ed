// Device-side helpers shared by the gfx950 kernels of the decoding hot path.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace brisk {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Low / high bf16 of a packed 32-bit word.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// ---------------------------------------------------------------------------
// Candidate keys.  A 64-bit key orders (logit descending, id ascending) as a
// plain unsigned integer: the high word is the float's bits made monotone,
// the low word is ~id.  The K largest keys are therefore exactly the ordered
// top-K, independent of the order in which keys are visited.  Key 0 is never
// produced by a finite logit and marks an empty slot.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t make_key(float logit, uint32_t id) {
  uint32_t u = __float_as_uint(logit + 0.0f);  // -0 -> +0
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<uint64_t>(u) << 32) | static_cast<uint64_t>(0xFFFFFFFFu - id);
}

__device__ __forceinline__ float key_logit(uint64_t key) {
  uint32_t u = static_cast<uint32_t>(key >> 32);
  u = (u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u;
  return __uint_as_float(u);
}

__device__ __forceinline__ int32_t key_id(uint64_t key) {
  return static_cast<int32_t>(0xFFFFFFFFu - static_cast<uint32_t>(key));
}

// Smallest logit that can still enter a list whose last entry is `last`
// (any finite logit while the list has an empty slot).  A logit equal to it
// may enter or not depending on its id, so callers compare with >=.
__device__ __forceinline__ float list_floor(uint64_t last) {
  return last == 0 ? -INFINITY : key_logit(last);
}

// Insert `key` into a list sorted descending, dropping the smallest entry.
// Branch-free: every slot keeps max(slot, carry) and passes min on.
template <int N>
__device__ __forceinline__ void list_insert(uint64_t (&list)[N], uint64_t key) {
#pragma unroll
  for (int j = 0; j < N; ++j) {
    const uint64_t hi = list[j] > key ? list[j] : key;
    const uint64_t lo = list[j] > key ? key : list[j];
    list[j] = hi;
    key = lo;
  }
}

// ---------------------------------------------------------------------------
// Wavefront reductions (64 lanes).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), off, kWave);
    const uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), off, kWave);
    const uint64_t o = (static_cast<uint64_t>(hi) << 32) | lo;
    v = o > v ? o : v;
  }
  return v;
}

// DPP all-reduce: four steps inside each 16-lane row (quad swaps, then the
// half-row and row mirrors pair up disjoint groups), then the four row totals
// are read out as wave-uniform scalars and combined in a fixed order.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ float row_sum16(float v) {
  v += dpp_f32<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f32<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_f32<0x141>(v);  // row_half_mirror
  v += dpp_f32<0x140>(v);  // row_mirror
  return v;
}

__device__ __forceinline__ float row_max16(float v) {
  v = fmaxf(v, dpp_f32<0xB1>(v));
  v = fmaxf(v, dpp_f32<0x4E>(v));
  v = fmaxf(v, dpp_f32<0x141>(v));
  v = fmaxf(v, dpp_f32<0x140>(v));
  return v;
}

template <int CTRL>
__device__ __forceinline__ int dpp_i32(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}

// v[lane] + v[lane ^ 16] and v[lane] + v[lane ^ 32] through the gfx950 lane
// swaps: the swap leaves a lane's own value in one result and its partner's
// in the other, and the sum is the same in both lanes of a pair.
__device__ __forceinline__ float swap16_sum(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float swap32_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float readlane_f32(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}

// Wave-uniform sum of v over the 64 lanes.
__device__ __forceinline__ float wave_allsum(float v) {
  v = row_sum16(v);
  return (readlane_f32(v, 0) + readlane_f32(v, 16)) + (readlane_f32(v, 32) + readlane_f32(v, 48));
}

// Wave-uniform maximum of v over the 64 lanes.
__device__ __forceinline__ float wave_allmax(float v) {
  v = row_max16(v);
  return fmaxf(fmaxf(readlane_f32(v, 0), readlane_f32(v, 16)), fmaxf(readlane_f32(v, 32), readlane_f32(v, 48)));
}

__device__ __forceinline__ float sigmoidf_(float x) { return 1.0f / (1.0f + __expf(-x)); }

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC'11): ten rounds of two
// 32x32 -> 64-bit products (multipliers 0xD2511F53, 0xCD9E8D57) and a Weyl
// key schedule (increments 0x9E3779B9, 0xBB67AE85).
// ---------------------------------------------------------------------------
// Each product is one 64-bit multiply-add (half the quarter-rate
// instructions of separate high and low halves).
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int i = 0; i < 10; ++i) {
    const uint64_t p0 = static_cast<uint64_t>(0xD2511F53u) * c.x;
    const uint64_t p1 = static_cast<uint64_t>(0xCD9E8D57u) * c.z;
    c = make_uint4(static_cast<uint32_t>(p1 >> 32) ^ c.y ^ k0, static_cast<uint32_t>(p1),
                   static_cast<uint32_t>(p0 >> 32) ^ c.w ^ k1, static_cast<uint32_t>(p0));
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// Gumbel variate of a generator word: U = (w / 512 + 1/2) / 2^23 lies
// strictly inside (0, 1) and is exact in single precision; G = -log(-log U),
// both logarithms from the hardware base-2 logarithm.  U >= 2^-24 and
// -log U >= 2^-24 are normal numbers, so it needs no subnormal scaling.
__device__ __forceinline__ float gumbel_of(uint32_t w) {
  constexpr float kLn2 = 0.69314718055994531f;
  const float U = (static_cast<float>(w >> 9) + 0.5f) * (1.0f / 8388608.0f);
  return -kLn2 * __builtin_amdgcn_logf(-kLn2 * __builtin_amdgcn_logf(U));
}

// Merge a log-sum-exp partial (max m, sum of exp(x - m)) into (m, s).
__device__ __forceinline__ void lse_combine(float& m, float& s, float2 o) {
  const float M = fmaxf(m, o.x);
  if (M == -INFINITY) return;
  s = s * __expf(m - M) + o.y * __expf(o.x - M);
  m = M;
}

__device__ __forceinline__ int clamp_id(int32_t id, int32_t V) {
  return id < 0 ? 0 : (id >= V ? V - 1 : id);
}

}  // namespace brisk
