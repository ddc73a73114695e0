// ss_device.hpp -- device primitives for the gfx950 sampler kernels.
//
// Order-preserving keys, Philox4x32-10, wave64 / workgroup reductions and
// scans, and an LDS bitonic sort.  Workgroups are kBlock = 512 threads
// (eight 64-lane wavefronts, two per SIMD).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ss {

constexpr int kBlock = 512;
constexpr int kWaves = kBlock / 64;
// the streaming launch (one unit per wavefront, plus the patch-table
// workgroups) keeps 256-thread workgroups
constexpr int kSBlock = 256;
constexpr int kSWaves = kSBlock / 64;

// ---------------------------------------------------------------------------
// Order-preserving 32-bit key of a float32 bit pattern.
//   positives  u  -> u + 2^31          (+0 -> 0x80000000)
//   negatives  u  -> 2^32 - u          (-0 -> 0x80000000: ties with +0)
// so key order is value order and -0 == +0.  -inf maps to kKeyNegInf,
// negative NaNs below it; positive NaNs (above +inf) are folded to 0.
// Keys <= kKeyNegInf are "invalid" (never selected).  The lexicographic
// encoding of the paper's Section 3.4 is the 16-bit analogue of this map.
// ---------------------------------------------------------------------------
constexpr uint32_t kKeyNegInf = 0x00800000u;
constexpr uint32_t kKeyPosInf = 0xFF800000u;
constexpr uint32_t kKeyFloor = kKeyNegInf + 1u;  // smallest valid key

__device__ __forceinline__ uint32_t key_of_bits(uint32_t u) {
  const uint32_t s = (uint32_t)((int32_t)u >> 31);
  const uint32_t k = (u ^ s) + (s ? 1u : 0x80000000u);
  return k > kKeyPosInf ? 0u : k;
}

__device__ __forceinline__ uint32_t key_of_float(float f) { return key_of_bits(__float_as_uint(f)); }

__device__ __forceinline__ float float_of_key(uint32_t k) {
  const uint32_t u = (k >= 0x80000000u) ? (k - 0x80000000u) : (0u - k);
  return __uint_as_float(u);
}

// canonical value of a logit: NaN -> -inf, -0 -> +0
__device__ __forceinline__ float canon(float v) {
  if (v != v) return -__builtin_inff();
  return v == 0.0f ? 0.0f : v;
}

// Composite rank key: larger = earlier in canonical order (value desc, index asc).
__device__ __forceinline__ uint64_t comp_of(uint32_t key, uint32_t idx) {
  return ((uint64_t)key << 32) | (uint64_t)(~idx);
}
__device__ __forceinline__ uint32_t comp_key(uint64_t c) { return (uint32_t)(c >> 32); }
__device__ __forceinline__ uint32_t comp_idx(uint64_t c) { return ~(uint32_t)c; }

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon et al., SC'11), counter (request, pos lo, pos hi, 0),
// key (seed lo, seed hi).  Word 0 drives token draws, word 1 acceptance.
// ---------------------------------------------------------------------------
__device__ inline uint4 philox4x32_10(uint4 c, uint2 k) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t hi0 = __umulhi(0xD2511F53u, c.x), lo0 = 0xD2511F53u * c.x;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c.z), lo1 = 0xCD9E8D57u * c.z;
    c = make_uint4(hi1 ^ c.y ^ k.x, lo1, hi0 ^ c.w ^ k.y, lo0);
    k.x += 0x9E3779B9u;
    k.y += 0xBB67AE85u;
  }
  return c;
}

__device__ inline double uniform01(uint64_t seed, uint32_t request, int64_t position, int word) {
  const uint64_t p = (uint64_t)position;
  const uint4 o = philox4x32_10(make_uint4(request, (uint32_t)p, (uint32_t)(p >> 32), 0u),
                                make_uint2((uint32_t)seed, (uint32_t)(seed >> 32)));
  const uint32_t w = word == 0 ? o.x : (word == 1 ? o.y : (word == 2 ? o.z : o.w));
  return ((double)w + 0.5) * (1.0 / 4294967296.0);
}

// weight of a kept token: exp((y - M)/tau), exactly 1 at the maximum
__device__ inline double weight_of(double y, double M, double tau) {
  return (y == M) ? 1.0 : exp((y - M) / tau);
}
// The same weight with the exponent (y - M) / tau formed in double and the
// exponential taken in float (about one ulp): relative error near 1e-7, far
// inside the 1e-5 relative agreement the probabilities are held to, at a
// fraction of the cost of a double exponential.
__device__ inline double weight_fast(double y, double M, double inv_tau) {
  return (y == M) ? 1.0 : (double)expf((float)((y - M) * inv_tau));
}

// ---------------------------------------------------------------------------
// wave64 / workgroup helpers
// ---------------------------------------------------------------------------

// Workgroup barrier that orders LDS only: global loads still in flight stay
// in flight (a full __syncthreads() fence is used only where global memory
// written by other threads must be ordered).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}
__device__ __forceinline__ int lane() { return (int)__lane_id(); }
__device__ __forceinline__ int wave() { return (int)(threadIdx.x >> 6); }

// ---------------------------------------------------------------------------
// Cross-lane primitives on DPP row operations (no LDS round trip).  Every
// lane of the wavefront must be active.  64-bit values move as two halves.
// ---------------------------------------------------------------------------
template <int CTRL, int ROWM = 0xF, int BANKM = 0xF, bool BC = false>
__device__ __forceinline__ uint32_t dpp32(uint32_t old, uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROWM, BANKM, BC);
}
template <int CTRL, int ROWM = 0xF, int BANKM = 0xF, bool BC = false>
__device__ __forceinline__ uint64_t dpp64(uint64_t old, uint64_t v) {
  const uint32_t lo = dpp32<CTRL, ROWM, BANKM, BC>((uint32_t)old, (uint32_t)v);
  const uint32_t hi = dpp32<CTRL, ROWM, BANKM, BC>((uint32_t)(old >> 32), (uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}
template <typename T, int CTRL, int ROWM = 0xF, int BANKM = 0xF, bool BC = false>
__device__ __forceinline__ T dppT(T old, T v) {
  if constexpr (sizeof(T) == 8) {
    return __builtin_bit_cast(T, dpp64<CTRL, ROWM, BANKM, BC>(__builtin_bit_cast(uint64_t, old),
                                                               __builtin_bit_cast(uint64_t, v)));
  } else {
    return __builtin_bit_cast(T, dpp32<CTRL, ROWM, BANKM, BC>(__builtin_bit_cast(uint32_t, old),
                                                               __builtin_bit_cast(uint32_t, v)));
  }
}
template <typename T>
__device__ __forceinline__ T readlane_T(T v, int l) {
  if constexpr (sizeof(T) == 8) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)u, l), hi = __builtin_amdgcn_readlane((uint32_t)(u >> 32), l);
    return __builtin_bit_cast(T, ((uint64_t)hi << 32) | lo);
  } else {
    return __builtin_bit_cast(T, (uint32_t)__builtin_amdgcn_readlane(__builtin_bit_cast(uint32_t, v), l));
  }
}
// every lane ends with the reduction over its 16-lane row
template <typename T, typename Op>
__device__ __forceinline__ T row_reduce(T v, Op op) {
  v = op(v, dppT<T, 0xB1>(v, v));   // quad_perm [1,0,3,2]
  v = op(v, dppT<T, 0x4E>(v, v));   // quad_perm [2,3,0,1]
  v = op(v, dppT<T, 0x141>(v, v));  // row_half_mirror
  v = op(v, dppT<T, 0x140>(v, v));  // row_mirror
  return v;
}
template <typename T, typename Op>
__device__ __forceinline__ T wave_reduce(T v, Op op) {
  v = row_reduce(v, op);
  return op(op(readlane_T(v, 0), readlane_T(v, 16)), op(readlane_T(v, 32), readlane_T(v, 48)));
}
template <typename T>
__device__ __forceinline__ T wave_max(T v) {
  return wave_reduce(v, [](T x, T y) { return x > y ? x : y; });
}
template <typename T>
__device__ __forceinline__ T wave_min(T v) {
  return wave_reduce(v, [](T x, T y) { return x < y ? x : y; });
}
template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
  return wave_reduce(v, [](T x, T y) { return x + y; });
}
// inclusive prefix sum over the 64 lanes: Hillis-Steele inside each row,
// then the row totals carried across rows
template <typename T>
__device__ __forceinline__ T wave_incl_scan(T v) {
  v += dppT<T, 0x111, 0xF, 0xF, true>(T(0), v);  // row_shr:1, zero fill
  v += dppT<T, 0x112, 0xF, 0xF, true>(T(0), v);  // row_shr:2
  v += dppT<T, 0x114, 0xF, 0xF, true>(T(0), v);  // row_shr:4
  v += dppT<T, 0x118, 0xF, 0xF, true>(T(0), v);  // row_shr:8
  v += dppT<T, 0x142, 0xA, 0xF, false>(T(0), v);  // row_bcast:15 into rows 1, 3
  v += dppT<T, 0x143, 0xC, 0xF, false>(T(0), v);  // row_bcast:31 into rows 2, 3
  return v;
}

// Workgroup reductions through a small LDS scratch of kWaves entries.
// Every call ends with a barrier so the scratch can be reused at once.
template <typename T>
__device__ inline T block_max(T v, T* scratch) {
  v = wave_max(v);
  if (lane() == 0) scratch[wave()] = v;
  lds_barrier();
  T r = scratch[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) r = scratch[w] > r ? scratch[w] : r;
  lds_barrier();
  return r;
}
template <typename T>
__device__ inline T block_min(T v, T* scratch) {
  v = wave_min(v);
  if (lane() == 0) scratch[wave()] = v;
  lds_barrier();
  T r = scratch[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) r = scratch[w] < r ? scratch[w] : r;
  lds_barrier();
  return r;
}
// Deterministic sum: fixed shuffle tree, then waves in order.
template <typename T>
__device__ inline T block_sum(T v, T* scratch) {
  v = wave_sum(v);
  if (lane() == 0) scratch[wave()] = v;
  lds_barrier();
  T r = scratch[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) r += scratch[w];
  lds_barrier();
  return r;
}
// Exclusive scan over threads in thread order; returns this thread's offset,
// writes the workgroup total.
template <typename T>
__device__ inline T block_excl_scan(T v, T* scratch, T& total) {
  const T inc = wave_incl_scan(v);
  if (lane() == 63) scratch[wave()] = inc;
  lds_barrier();
  T off = T(0), tot = T(0);
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const T s = scratch[w];
    if (w < wave()) off += s;
    tot += s;
  }
  lds_barrier();
  total = tot;
  return off + inc - v;
}

// ---------------------------------------------------------------------------
// LDS bitonic sort, descending, of n (power of two) 64-bit keys.
// ---------------------------------------------------------------------------
__device__ inline void lds_sort_desc(uint64_t* a, int n) {
  for (int k = 2; k <= n; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int p = threadIdx.x; p < (n >> 1); p += kBlock) {
        const int i = ((p & ~(j - 1)) << 1) | (p & (j - 1));
        const int m = i + j;
        const uint64_t x = a[i], y = a[m];
        const bool desc = (i & k) == 0;
        if (desc ? (x < y) : (x > y)) {
          a[i] = y;
          a[m] = x;
        }
      }
      lds_barrier();
    }
  }
}


// ---------------------------------------------------------------------------
// wave64 helpers built on DPP row operations and ballots (no LDS traffic).
// Every lane of the wavefront must be active.
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}
// maximum over the wavefront, returned in a scalar register
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  v = max(v, dpp_mov<0xB1>(v));   // quad_perm [1,0,3,2]
  v = max(v, dpp_mov<0x4E>(v));   // quad_perm [2,3,0,1]
  v = max(v, dpp_mov<0x141>(v));  // row_half_mirror
  v = max(v, dpp_mov<0x140>(v));  // row_mirror: every lane holds its row's maximum
  const uint32_t r0 = __builtin_amdgcn_readlane(v, 0), r1 = __builtin_amdgcn_readlane(v, 16);
  const uint32_t r2 = __builtin_amdgcn_readlane(v, 32), r3 = __builtin_amdgcn_readlane(v, 48);
  return max(max(r0, r1), max(r2, r3));
}
// exclusive prefix over lanes of small per-lane counts c < 32 (bit planes
// counted with mbcnt); `total` receives the wavefront sum
__device__ __forceinline__ uint32_t wave_excl_small(uint32_t c, uint32_t& total) {
  uint32_t off = 0u, tot = 0u;
#pragma unroll
  for (int b = 0; b < 5; ++b) {
    const uint64_t m = __ballot((c >> b) & 1u);
    off += __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u)) << b;
    tot += (uint32_t)__popcll(m) << b;
  }
  total = tot;
  return off;
}

__host__ __device__ inline int next_pow2(int v) {
  int p = 1;
  while (p < v) p <<= 1;
  return p;
}

}  // namespace ss
