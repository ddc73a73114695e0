// ss_kernel.hip -- fused LLM sampling pipeline for MI355X (gfx950).
//
// One launch per call (plus one materialising pass for ss_process_logits).
// Grid: rows x T workgroups, T = ceil(V / kTile).  Each workgroup streams one
// kTile-element slice of one logit row exactly once and
//   1. applies the logit-processing prologue (paper Appendix C.1, Alg. 8
//      order): grammar allow bits, repetition / frequency / presence penalties
//      and sparse logit bias -- penalties and bias touch only the ids in the
//      request's history / bias lists, so they are computed once per distinct
//      id by an "owner" thread and the bulk of the tile pays nothing for them;
//   2. turns every element into an order-preserving 32-bit key;
//   3. reduces the tile maximum (greedy rows stop here);
//   4. for truncating rows, derives an emission threshold from the maxima of
//      groups of 4 elements (the q-th largest group maximum bounds the tile's
//      q-th largest element from below) and writes the elements at or above
//      it to a small per-tile candidate region -- a bounded candidate set, as
//      in the paper's two-stage scheme (Section 3.2), but with a row-level
//      quota instead of a fixed per-tile k;
//   5. takes a ticket; the last workgroup of the row merges: it checks that
//      the candidates provably contain the row's top-k (at least k of them lie
//      above the largest tile threshold), selects the exact top-k by radix
//      select in registers, and runs the truncation / selection epilogue
//      (Alg. 11 order) in double precision.  If the check fails (skewed or
//      heavily tied rows) it recomputes the exact top-k by streaming the row
//      again -- a slow but always-correct path, flagged SS_FLAG_FALLBACK.
// No host synchronisation, fixed grid, self-resetting counters: every call
// can be captured in a HIP graph.
#include <hip/hip_runtime.h>
#include <limits.h>
#include <stddef.h>
#include <stdint.h>

#include "ss.h"
#include "ss_device.hpp"

namespace ss {

constexpr int kTile = 8192;
constexpr int kPT = kTile / kBlock;  // element slots per thread (32)
constexpr int kGPT = 8;              // group maxima per thread
constexpr int kGS = kPT / kGPT;      // slots per group (4)
constexpr int kUnits = kWaves;       // emission units per tile: one per wavefront
constexpr int kUnitElems = kTile / kUnits;  // elements per unit (2048)
constexpr int kUnitGroups = kGPT * 64;      // group maxima per unit (512)
constexpr int kHCap = 1024;          // in-tile history entries held in LDS
constexpr int kBCap = 128;           // in-tile bias entries held in LDS
constexpr int kPCap = 128;           // patched slots per wavefront held in LDS
constexpr int kIdsPT = 2;            // history ids each thread loads up front
constexpr int kRPT = 32;             // merge candidates per thread (registers)
constexpr int kMaxT = (SS_MAX_V + kTile - 1) / kTile;
constexpr int kMaxU = kMaxT * kUnits;  // emission units per row
constexpr int kEPT = SS_MAX_K / kBlock;  // selected entries per thread in the epilogue
constexpr int kHCopies = 4;              // privatised histogram copies (lane & 3)
constexpr int kHStride = 257;            // padded so copies of one bin sit in different banks
constexpr uint32_t kNoEmit = 0xFFFFFFFFu;  // emits nothing (above every valid key)
constexpr double kFix = 1125899906842624.0;  // 2^50: fixed-point scale of weight sums

enum { OP_TOPK = SS_OP_TOPK, OP_SAMPLE = SS_OP_SAMPLE, OP_VERIFY = SS_OP_VERIFY, OP_PROCESS = SS_OP_PROCESS };
enum { KIND_EMPTY = 0, KIND_GREEDY = 1, KIND_DIST = 2 };

struct RowSummary {
  uint64_t thr;  // composite key of the last kept rank
  double Z;      // sum of kept weights
  float M;       // row maximum
  float tau;
  int32_t argmax;
  int32_t kind;
};
struct RowResult {
  int32_t accept;
  int32_t emit;
  int32_t flags;
  int32_t pad;
};

struct KArgs {
  const void* x;
  int64_t ld;
  int op, B, rows, V, T, L, k_cap, cap, k_out, vec_ok;
  uint32_t feat;
  const uint32_t* mode;
  const float* temperature;
  const int32_t* top_k;
  const float* top_p;
  const float* min_p;
  const float* rep;
  const float* freq;
  const float* pres;
  const int32_t* hist_off;
  const int32_t* hist_ids;
  const int32_t* bias_off;
  const int32_t* bias_ids;
  const float* bias_vals;
  const uint32_t* bitmask;
  int64_t mask_ld;
  const uint64_t* seed;
  const int64_t* position;
  const float* draft_probs;
  int64_t ld_q;
  const int32_t* draft_tokens;
  int32_t* out_token;
  float* out_logprob;
  int32_t* out_idx;
  float* out_prob;
  int32_t* flags;
  float* out_val;
  int32_t* out_tokens;
  int32_t* out_nacc;
  float* out_logits;
  float* out_probs;
  uint32_t* ticket;
  uint32_t* req_ticket;
  uint4* rec;
  uint2* cand;
  RowResult* res;
  RowSummary* summ;
};

// ---------------------------------------------------------------------------
// Per-row context
// ---------------------------------------------------------------------------
struct Ctx {
  int row, req, ell;
  uint32_t mode;
  const unsigned char* xrow;
  const int32_t* hist;
  int nhist;
  const int32_t* extra;
  int nextra;
  const int32_t* bias_ids;
  const float* bias_vals;
  int nbias;
  const uint32_t* mask;
  float rep, freq, pres;
  bool greedy;
  bool kcap;
  int k_eff;
};

struct Smem {
  uint64_t red64[kWaves];
  double redd[kWaves];
  double bcd[4];
  uint2 pw[kWaves][kPCap];  // per-wave patched slots: (lane | slot<<6 | bias<<11 | count<<12, bias sum)
  uint32_t bm[kBlock];      // per-thread bits of patched slots
  int32_t bl_pos[kBCap];
  float bl_val[kBCap];
  uint32_t prefix[kMaxU + 1];
  uint32_t pw_n[kWaves];
  uint32_t red32[kWaves];
  uint32_t cnt[4];
  uint32_t bc[8];
  uint16_t hl[kHCap];  // distinct history ids of the tile (local index)
  uint16_t bl_l[kBCap];
  uint32_t cnt8[kTile / 4];     // packed 8-bit occurrence counts per local index
  // merge only from here
  uint32_t hist[2][kHCopies * kHStride];  // double-buffered privatised radix histograms
  uint32_t low[2][64];  // per bin (bytes): some key in the bin has non-zero bits below the digit
  KArgs fa;              // kernel arguments and row context handed to the fallback
  Ctx fc;
};
constexpr int kSmemStream = (int)((offsetof(Smem, hist) + 15) & ~(size_t)15);
constexpr int kSmemFixed = (int)((sizeof(Smem) + 15) & ~(size_t)15);
// merge dynamic LDS: [Smem][candidates: kRPT * kBlock uint2][sel: next_pow2(k_max) uint64]
constexpr int kCandBytes = 8 * kRPT * kBlock;
constexpr int kSelOff = kSmemFixed + kCandBytes;

// ---------------------------------------------------------------------------
// Element layout: thread t, slot j (0..31) holds chunk i = j / VW, element
// e = j % VW of vector v = i * kBlock + t, i.e. local index (v * VW + e).
// A chunk is one 16-byte load (8 bf16 or 4 float32).
// ---------------------------------------------------------------------------
template <int DT>
struct DTT;
template <>
struct DTT<SS_F32> {
  static constexpr int VW = 4, NV = 8, ES = 4;
};
template <>
struct DTT<SS_BF16> {
  static constexpr int VW = 8, NV = 4, ES = 2;
};

template <int DT>
__device__ __forceinline__ int local_of_slot(int t, int j) {
  constexpr int VW = DTT<DT>::VW;
  return ((j / VW) * kBlock + t) * VW + (j % VW);
}

// key without the positive-NaN fold; callers fold when the maximum exceeds +inf
__device__ __forceinline__ uint32_t key_raw(uint32_t u) {
  const uint32_t s = (uint32_t)((int32_t)u >> 31);
  return (u ^ s) + (s ? 1u : 0x80000000u);
}
__device__ __forceinline__ uint32_t fold_nan(uint32_t k) { return k > kKeyPosInf ? 0u : k; }

__device__ __forceinline__ uint32_t comp4(const uint4& v, int c) {
  return c == 0 ? v.x : (c == 1 ? v.y : (c == 2 ? v.z : v.w));
}

// float32 bit pattern of slot j
template <int DT>
__device__ __forceinline__ uint32_t slot_bits(const uint4 (&r)[DTT<DT>::NV], int j) {
  if constexpr (DT == SS_F32) {
    return comp4(r[j >> 2], j & 3);
  } else {
    const uint32_t w = comp4(r[j >> 3], (j & 7) >> 1);
    return (j & 1) ? (w & 0xFFFF0000u) : (w << 16);
  }
}

// raw element load from global memory (scalar), as float32 bits
template <int DT>
__device__ __forceinline__ uint32_t load_elem_bits(const unsigned char* xrow, int64_t i) {
  if constexpr (DT == SS_F32) {
    return reinterpret_cast<const uint32_t*>(xrow)[i];
  } else {
    return ((uint32_t)reinterpret_cast<const uint16_t*>(xrow)[i]) << 16;
  }
}


template <int DT>
__device__ __forceinline__ Ctx make_ctx(const KArgs& a, int row) {
  Ctx c;
  c.row = row;
  if (a.op == OP_VERIFY) {
    c.req = row / (a.L + 1);
    c.ell = row % (a.L + 1);
  } else {
    c.req = row;
    c.ell = 0;
  }
  const int b = c.req;
  const uint32_t m = (a.op == OP_TOPK ? SS_TOPK : (a.mode ? a.mode[b] : 0u)) & a.feat;
  c.mode = m;
  c.xrow = reinterpret_cast<const unsigned char*>(a.x) + (size_t)row * (size_t)a.ld * DTT<DT>::ES;
  c.hist = nullptr;
  c.nhist = 0;
  c.extra = nullptr;
  c.nextra = 0;
  if (m & (SS_REP | SS_FREQ | SS_PRES)) {
    c.hist = a.hist_ids + a.hist_off[b];
    c.nhist = a.hist_off[b + 1] - a.hist_off[b];
    if (a.op == OP_VERIFY && a.draft_tokens) {
      c.extra = a.draft_tokens + (size_t)b * a.L;
      c.nextra = c.ell;
    }
  }
  c.bias_ids = nullptr;
  c.bias_vals = nullptr;
  c.nbias = 0;
  if (m & SS_BIAS) {
    c.bias_ids = a.bias_ids + a.bias_off[b];
    c.bias_vals = a.bias_vals + a.bias_off[b];
    c.nbias = a.bias_off[b + 1] - a.bias_off[b];
  }
  c.mask = (m & SS_GRAMMAR) ? a.bitmask + (size_t)row * (size_t)a.mask_ld : nullptr;
  c.rep = (m & SS_REP) ? a.rep[b] : 1.0f;
  c.freq = (m & SS_FREQ) ? a.freq[b] : 0.0f;
  c.pres = (m & SS_PRES) ? a.pres[b] : 0.0f;
  c.kcap = false;
  if (a.op == OP_TOPK) {
    c.greedy = false;
    int k = a.top_k ? a.top_k[b] : a.k_cap;
    c.k_eff = k < 0 ? 0 : (k > a.k_cap ? a.k_cap : k);
  } else {
    c.greedy = (m & SS_GREEDY) || ((m & SS_TEMP) && a.temperature[b] <= 0.0f);
    const int64_t kreq = ((m & SS_TOPK) && a.top_k[b] >= 1) ? (int64_t)a.top_k[b] : (int64_t)INT_MAX;
    c.k_eff = kreq < a.k_cap ? (int)kreq : a.k_cap;
    c.kcap = !c.greedy && kreq > a.k_cap;
  }
  return c;
}

// Candidate quota of one emission unit when a row's top-k is spread over U
// units: the unit emits at least its q largest elements (by its threshold),
// with q well above the unit's expected share k/U, so that the largest unit
// threshold lies below the row's k-th value except with tiny probability.
__host__ __device__ inline int quota(int k, int U) {
  if (U <= 1) return k;
  const int kt = (k + U - 1) / U;
  int s = 0;
  while (s * s < kt) ++s;
  const int q = kt + 5 * s + 6;
  return q < k ? q : k;
}

// capacity of one unit's candidate region
__host__ __device__ inline int unit_cap(int kcap, int U) {
  const int q = quota(kcap, U);
  if (2 * q > kUnitGroups) return kUnitElems;
  const int c = 2 * q + 32;
  return c < kUnitElems ? c : kUnitElems;
}

// ---------------------------------------------------------------------------
// Prologue of one element in Appendix C.1 order, each step one float32 op:
// repetition penalty, frequency and presence penalties (count > 0), then the
// logit bias.  Grammar masking is applied by the caller.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t penalised_key(uint32_t bits, uint32_t mode, float rep, float freq, float pres,
                                                  int count, bool has_bias, float bsum) {
  float v = canon(__uint_as_float(bits));
  if (count > 0) {
    if (mode & SS_REP) v = (v > 0.0f) ? v / rep : v * rep;
    if (mode & SS_FREQ) {
      const float t = freq * (float)count;
      v = v - t;
    }
    if (mode & SS_PRES) v = v - pres;
  }
  if (has_bias) v = v + bsum;
  return key_of_float(v);
}

template <int DT>
__device__ __forceinline__ void slot_of_local(int l, int* t, int* j) {
  constexpr int VW = DTT<DT>::VW;
  const int v = l / VW, e = l % VW;
  *t = v % kBlock;
  *j = (v / kBlock) * VW + e;
}

template <int DT>
__device__ __forceinline__ void set_patch_bit(Smem& S, int l) {
  int t, j;
  slot_of_local<DT>(l, &t, &j);
  atomicOr(&S.bm[t], 1u << j);
}

// float32 bits of raw slot j for a wave-uniform j: the chunk registers are
// viewed as one vector so the uniform index becomes register-relative moves.
typedef uint32_t u32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x32 __attribute__((ext_vector_type(32)));
template <int DT>
__device__ __forceinline__ uint32_t slot_bits_uniform(const uint4 (&r)[DTT<DT>::NV], int j) {
  if constexpr (DT == SS_F32) {
    u32x32 v;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      v[4 * q + 0] = r[q].x;
      v[4 * q + 1] = r[q].y;
      v[4 * q + 2] = r[q].z;
      v[4 * q + 3] = r[q].w;
    }
    return v[j];
  } else {
    u32x16 v;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      v[4 * q + 0] = r[q].x;
      v[4 * q + 1] = r[q].y;
      v[4 * q + 2] = r[q].z;
      v[4 * q + 3] = r[q].w;
    }
    const uint32_t w = v[j >> 1];
    return (j & 1) ? (w & 0xFFFF0000u) : (w << 16);
  }
}

// ---------------------------------------------------------------------------
// Loads one tile and produces the processed keys of this thread's 32 slots
// (0 = invalid: masked, NaN, beyond V).  The request's history / bias ids are
// fetched before the tile so that building the in-tile patch lists overlaps
// the tile's own loads; one owner per distinct id computes its occurrence
// count and ordered bias sum from LDS, and the thread holding that element
// applies the penalties to its registers.  Long lists that overflow LDS fall
// back to per-slot scans of the global lists (rare, exact).
// ---------------------------------------------------------------------------
template <int DT, bool FULL>
__device__ __forceinline__ void load_tile(const KArgs& a, const Ctx& c, int lo, Smem& S, uint32_t (&key)[kPT]) {
  constexpr int VW = DTT<DT>::VW, NV = DTT<DT>::NV, ES = DTT<DT>::ES;
  const int tid = threadIdx.x;
  const int V = a.V;
  const int n_tile = min(kTile, V - lo);
  const bool do_hist = (c.mode & (SS_REP | SS_FREQ | SS_PRES)) && (c.nhist + c.nextra) > 0;
  const bool do_bias = (c.mode & SS_BIAS) && c.nbias > 0;
  const bool patch = do_hist || do_bias;
  const int nh = c.nhist + c.nextra;

  // 1. request lists and grammar words first, as a fixed sequence of loads
  //    (disabled entries read a dummy in-bounds address), so that waiting for
  //    them never has to drain the tile loads issued after them.
  const int32_t* dummy = reinterpret_cast<const int32_t*>(c.xrow);
  int hid[kIdsPT];
#pragma unroll
  for (int u = 0; u < kIdsPT; ++u) {
    const int h = tid + u * kBlock;
    const bool ok = do_hist && h < nh;
    const int32_t* src = !ok ? dummy : (h < c.nhist ? c.hist + h : c.extra + (h - c.nhist));
    hid[u] = *src;
    if (!ok) hid[u] = -1;
  }
  const bool bok = do_bias && tid < c.nbias;
  int bid = *(bok ? c.bias_ids + tid : dummy);
  float bval = *(bok ? c.bias_vals + tid : reinterpret_cast<const float*>(dummy));
  if (!bok) bid = -1;
  uint32_t mw[NV];
  {
    const int W = (V + 31) >> 5;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int wi = (lo + (i * kBlock + tid) * VW) >> 5;
      const bool ok = c.mask != nullptr && wi < W;
      mw[i] = *(ok ? c.mask + wi : reinterpret_cast<const uint32_t*>(dummy));
      if (!ok) mw[i] = 0u;
    }
  }

  // 2. the tile
  uint4 raw[NV];
  if constexpr (FULL) {
    // full, aligned tile: all 16-byte loads in flight together
    const uint4* src = reinterpret_cast<const uint4*>(c.xrow + (size_t)lo * ES);
#pragma unroll
    for (int i = 0; i < NV; ++i) raw[i] = src[i * kBlock + tid];
  } else {
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int l0 = (i * kBlock + tid) * VW;
    if (a.vec_ok && l0 + VW <= n_tile) {
      raw[i] = *reinterpret_cast<const uint4*>(c.xrow + ((size_t)lo + l0) * ES);
    } else {
      uint32_t w[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) w[q] = 0xFFFFFFFFu;  // negative NaN: invalid
#pragma unroll
      for (int e = 0; e < VW; ++e) {
        const int l = l0 + e;
        if (l < n_tile) {
          if constexpr (DT == SS_F32) {
            w[e] = reinterpret_cast<const uint32_t*>(c.xrow)[lo + l];
          } else {
            const uint32_t h = reinterpret_cast<const uint16_t*>(c.xrow)[lo + l];
            const int q = e >> 1;
            w[q] = (e & 1) ? ((w[q] & 0x0000FFFFu) | (h << 16)) : ((w[q] & 0xFFFF0000u) | h);
          }
        }
      }
      raw[i] = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
  }
  // 3. in-tile patch lists and owners (LDS only; overlaps the tile loads).
  //    Occurrences are counted in a packed 8-bit table; the entry whose
  //    increment finds zero owns the id and records it once.  A count that
  //    would pass 255 sends the tile to the exact slow path.
  bool overflow = false;
  if (patch) {
    S.bm[tid] = 0u;
    if (tid < 4) S.cnt[tid] = 0u;
    if (tid < kWaves) S.pw_n[tid] = 0u;
#pragma unroll
    for (int q = 0; q < kTile / 4 / kBlock / 4; ++q)
      reinterpret_cast<uint4*>(S.cnt8)[q * kBlock + tid] = make_uint4(0u, 0u, 0u, 0u);
    lds_barrier();
    auto add_hist = [&](int id) {
      const int rel = id - lo;
      if (id >= 0 && id < V && rel >= 0 && rel < n_tile) {
        const uint32_t sh = (uint32_t)(rel & 3) * 8u;
        const uint32_t old = (atomicAdd(&S.cnt8[rel >> 2], 1u << sh) >> sh) & 0xFFu;
        if (old == 0xFFu) S.cnt[2] = 1u;  // saturated
        if (old == 0u) {
          const uint32_t p = atomicAdd(&S.cnt[0], 1u);
          if (p < (uint32_t)kHCap) S.hl[p] = (uint16_t)rel;
          set_patch_bit<DT>(S, rel);
        }
      }
    };
#pragma unroll
    for (int u = 0; u < kIdsPT; ++u) add_hist(hid[u]);
    for (int h = tid + kIdsPT * kBlock; h < nh; h += kBlock)  // long histories
      add_hist(h < c.nhist ? c.hist[h] : c.extra[h - c.nhist]);
    auto add_bias = [&](int e, int id, float val) {
      const int rel = id - lo;
      if (id >= 0 && id < V && rel >= 0 && rel < n_tile) {
        const uint32_t p = atomicAdd(&S.cnt[1], 1u);
        if (p < (uint32_t)kBCap) {
          S.bl_l[p] = (uint16_t)rel;
          S.bl_pos[p] = e;
          S.bl_val[p] = val;
        }
        set_patch_bit<DT>(S, rel);
      }
    };
    if (do_bias && tid < c.nbias) add_bias(tid, bid, bval);
    for (int e = tid + kBlock; e < c.nbias; e += kBlock) add_bias(e, c.bias_ids[e], c.bias_vals[e]);
    lds_barrier();
    const int hl_n = (int)S.cnt[0], bl_n = (int)S.cnt[1];
    overflow = hl_n > kHCap || bl_n > kBCap || S.cnt[2] != 0u;
    if (!overflow) {
      for (int n = tid; n < hl_n + bl_n; n += kBlock) {
        int l;
        bool owner = true;
        if (n < hl_n) {
          l = S.hl[n];
        } else {
          const int nb = n - hl_n;
          l = S.bl_l[nb];
          // ids with a history count are owned by their history entry
          owner = ((S.cnt8[l >> 2] >> ((l & 3) * 8)) & 0xFFu) == 0u;
          for (int m = 0; m < nb && owner; ++m)
            if (S.bl_l[m] == l) owner = false;
        }
        if (!owner) continue;
        const int cntv = (int)((S.cnt8[l >> 2] >> ((l & 3) * 8)) & 0xFFu);
        float bsum = 0.0f;
        bool hb = false;
        if (do_bias) {
          int last = -1;
          for (;;) {  // this id's entries in list order
            int best = INT_MAX, bi = -1;
            for (int m = 0; m < bl_n; ++m)
              if (S.bl_l[m] == l && S.bl_pos[m] > last && S.bl_pos[m] < best) {
                best = S.bl_pos[m];
                bi = m;
              }
            if (bi < 0) break;
            bsum = bsum + S.bl_val[bi];
            hb = true;
            last = best;
          }
        }
        int t, j;
        slot_of_local<DT>(l, &t, &j);
        const int w = t >> 6;
        const uint32_t p = atomicAdd(&S.pw_n[w], 1u);
        if (p < (uint32_t)kPCap)
          S.pw[w][p] = make_uint2((uint32_t)(t & 63) | ((uint32_t)j << 6) | ((hb ? 1u : 0u) << 11) |
                                      ((uint32_t)cntv << 12),
                                  __float_as_uint(bsum));
      }
      lds_barrier();
#pragma unroll
      for (int w = 0; w < kWaves; ++w) overflow = overflow || S.pw_n[w] > (uint32_t)kPCap;
    }
  }

  // 4. keys (grammar allow bits first: one per slot); the keys live in one
  //    vector so a patched slot can be written with a wave-uniform index
  uint32_t allow = 0xFFFFFFFFu;
  if (c.mask) {
    allow = 0u;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int g0 = lo + (i * kBlock + tid) * VW;
      allow |= ((mw[i] >> (g0 & 31)) & ((1u << VW) - 1u)) << (i * VW);
    }
  }
  u32x32 kv;
  if (c.mask) {
#pragma unroll
    for (int j = 0; j < kPT; ++j) {
      const uint32_t k = key_raw(slot_bits<DT>(raw, j));
      kv[j] = ((allow >> j) & 1u) ? k : 0u;
    }
  } else {
#pragma unroll
    for (int j = 0; j < kPT; ++j) kv[j] = key_raw(slot_bits<DT>(raw, j));
  }

  // 5. penalties / bias: the holder of each patched slot rewrites its key
  if (patch && !overflow) {
    const int w = wave();
    const int n = (int)S.pw_n[w];
    for (int e = 0; e < n; ++e) {
      const uint2 ent = S.pw[w][e];
      const uint32_t hdr = __builtin_amdgcn_readfirstlane(ent.x);
      const int slot = (int)((hdr >> 6) & 31u);
      const uint32_t bits = slot_bits_uniform<DT>(raw, slot);
      if (lane() == (int)(hdr & 63u) && ((allow >> slot) & 1u)) {
        kv[slot] = penalised_key(bits, c.mode, c.rep, c.freq, c.pres, (int)(hdr >> 12), ((hdr >> 11) & 1u) != 0u,
                                 __uint_as_float(__builtin_amdgcn_readfirstlane(ent.y)));
      }
    }
  }
#pragma unroll
  for (int j = 0; j < kPT; ++j) key[j] = kv[j];
  if (patch && overflow) {
    const uint32_t pbits = S.bm[tid];
#pragma unroll
    for (int j = 0; j < kPT; ++j) {
      if ((pbits >> j) & 1u) {
        const int id = lo + local_of_slot<DT>(tid, j);
        int cntv = 0;
        if (do_hist) {
          for (int h = 0; h < c.nhist; ++h) cntv += (c.hist[h] == id);
          for (int h = 0; h < c.nextra; ++h) cntv += (c.extra[h] == id);
        }
        float bsum = 0.0f;
        bool hb = false;
        if (do_bias) {
          for (int e = 0; e < c.nbias; ++e)
            if (c.bias_ids[e] == id) {
              bsum = bsum + c.bias_vals[e];
              hb = true;
            }
        }
        if ((allow >> j) & 1u)
          key[j] = penalised_key(slot_bits<DT>(raw, j), c.mode, c.rep, c.freq, c.pres, cntv, hb, bsum);
      }
    }
  }
  if (patch) lds_barrier();  // LDS lists may be rebuilt by the caller's next tile
}

// A tile takes the straight-line path when it is complete and 16-byte aligned.
__device__ __forceinline__ bool tile_full(const KArgs& a, int lo) { return a.vec_ok && a.V - lo >= kTile; }

// ---------------------------------------------------------------------------
// Radix selection in the merge.  Histograms are privatised (kHCopies copies,
// stride kHStride) and double-buffered: the buffer of the next pass is
// cleared while the current one fills, so one barrier separates passes.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void radix_clear(Smem& S, int buf) {
  for (int i = threadIdx.x; i < kHCopies * kHStride; i += kBlock) S.hist[buf][i] = 0u;
  if (threadIdx.x < 64) S.low[buf][threadIdx.x] = 0u;
}
__device__ __forceinline__ void hist_add(uint32_t* h, uint32_t bin, bool pred) {
  if (pred) atomicAdd(&h[(lane() & (kHCopies - 1)) * kHStride + bin], 1u);
}
__device__ __forceinline__ void low_mark(uint32_t* low, uint32_t bin, bool pred) {
  if (pred) reinterpret_cast<uint8_t*>(low)[bin] = 1;
}

// Digit search by wave 0 over nb <= 256 bins.  Descending: find d with
// above(d) < want <= above(d) + h[d], above(d) = count in the bins above d;
// ascending: the same with the bins below d.  Writes (d, count before d, h[d],
// low flag of d) to bc[0..3]; d = nb if the total is below `want`.
__device__ inline void radix_digit(const uint32_t* h, const uint32_t* low, int nb, uint32_t want, bool descending,
                                   uint32_t* bc) {
  if (threadIdx.x < 64) {
    const int l = lane();
    uint32_t cb[4];
    uint32_t s = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = 4 * l + u;
      const int bin = descending ? (nb - 1 - r) : r;
      uint32_t v = 0;
      if (r < nb) {
#pragma unroll
        for (int cp = 0; cp < kHCopies; ++cp) v += h[cp * kHStride + bin];
      }
      cb[u] = v;
      s += v;
    }
    const uint32_t inc = wave_incl_scan(s);
    const uint32_t total = __shfl(inc, 63, 64);
    uint32_t run = inc - s;
    if (l == 0) {
      bc[0] = (uint32_t)nb;
      bc[1] = total;
      bc[2] = 0u;
      bc[3] = 1u;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = 4 * l + u;
      const int bin = descending ? (nb - 1 - r) : r;
      if (r < nb && run < want && run + cb[u] >= want) {
        bc[0] = (uint32_t)bin;
        bc[1] = run;
        bc[2] = cb[u];
        bc[3] = low ? (low[bin >> 2] >> (8 * (bin & 3))) & 255u : 1u;
      }
      run += cb[u];
    }
  }
  lds_barrier();
}

// ---------------------------------------------------------------------------
// Exact selection of the `want` largest composites (key desc, index asc)
// among the n_valid valid keys a visitor produces.  visit(f) calls f(key, idx)
// for this thread's elements; every thread calls it the same number of times.
// Every valid visited key lies in [lo_key, hi_key]: the bits above the
// highest bit in which the two bounds differ are common to all of them, so
// the 8-bit digit passes start just below those bits (first_window).  A pass
// whose chosen bin holds only keys with zero bits below the digit fixes the
// boundary key at once (bf16 logits leave the low 16 bits zero).  Ties at the
// boundary key take the lowest indices (indices < V): by direct ranking when
// there are at most kBlock of them, else by index digit passes.  With
// first_built the caller has already filled radix buffer 0 with the first
// key pass; otherwise buffer 0 must be cleared and published.  Returns
// (tk, ti): an element is selected iff key > tk or (key == tk and idx <= ti).
// ---------------------------------------------------------------------------
struct Window {
  int sh;       // shift of the first digit
  uint32_t dm;  // digit mask of the first pass
};
__device__ __forceinline__ Window first_window(uint32_t lo_key, uint32_t hi_key) {
  const int sh = 32 - __clz(lo_key ^ hi_key);
  const int w = sh < 8 ? sh : 8;
  return Window{sh - w, (1u << w) - 1u};
}

template <typename Visit>
__device__ __forceinline__ void radix_select(Visit&& visit, uint32_t want, uint32_t n_valid, uint32_t lo_key,
                                             uint32_t hi_key, int V, bool first_built, Smem& S, uint32_t* tk_out,
                                             uint32_t* ti_out) {
  int cur = 0;
  int sh = 32 - __clz(lo_key ^ hi_key);  // bits [0, sh) vary among the keys
  uint32_t prefix = sh >= 32 ? 0u : (hi_key >> sh);
  uint32_t tk = hi_key, ti = 0xFFFFFFFFu;
  uint32_t n_tie = n_valid;
  bool ties = true;
  bool skip_visit = first_built;
  if (want >= n_valid) {  // everything valid is selected
    tk = kKeyNegInf;
    ties = false;
    sh = 0;
  }
  while (sh > 0) {
    const int w = sh < 8 ? sh : 8;
    sh -= w;
    const int hs = sh + w;
    const uint32_t dm = (1u << w) - 1u;
    const uint32_t lm = (1u << sh) - 1u;
    uint32_t* h = S.hist[cur];
    uint32_t* lw = S.low[cur];
    if (!skip_visit) {
      visit([&](uint32_t k, uint32_t) {
        const bool part = k >= kKeyFloor && (hs >= 32 || (k >> hs) == prefix);
        const uint32_t d = (k >> sh) & dm;
        hist_add(h, d, part);
        low_mark(lw, d, part && (k & lm) != 0u);
      });
    }
    skip_visit = false;
    radix_clear(S, cur ^ 1);
    lds_barrier();
    radix_digit(h, lw, (int)dm + 1, want, true, S.bc);
    const uint32_t d = S.bc[0], above = S.bc[1], hd = S.bc[2], lowd = S.bc[3];
    cur ^= 1;
    if (d > dm) {  // fewer valid keys than `want`: all are selected
      tk = kKeyNegInf;
      ti = 0xFFFFFFFFu;
      ties = false;
      break;
    }
    prefix = (prefix << w) | d;
    want -= above;
    if (hd == want) {  // every key with this prefix is selected
      tk = prefix << sh;
      ti = 0xFFFFFFFFu;
      ties = false;
      break;
    }
    if (sh == 0 || lowd == 0u) {  // the boundary keys all equal prefix << sh
      tk = prefix << sh;
      n_tie = hd;
      break;
    }
  }
  if (ties && n_tie <= (uint32_t)kBlock) {
    // few ties: list their indices, rank each against the others
    uint32_t cnt = 0;
    visit([&](uint32_t k, uint32_t) { cnt += k == tk ? 1u : 0u; });
    uint32_t tot;
    uint32_t off = block_excl_scan(cnt, S.red32, tot);
    uint32_t* tl = S.hist[cur];  // free: cleared for a next pass that does not come
    visit([&](uint32_t k, uint32_t i) {
      if (k == tk) tl[off++] = i;
    });
    lds_barrier();
    if (threadIdx.x < tot) {
      const uint32_t my = tl[threadIdx.x];
      uint32_t r = 0;
      for (uint32_t j = 0; j < tot; ++j) r += tl[j] < my ? 1u : 0u;
      if (r == want - 1u) S.bc[4] = my;
    }
    lds_barrier();
    ti = S.bc[4];
  } else if (ties) {
    // many ties: the `want` lowest indices by index digit passes
    if (skip_visit) {  // no key pass ran: buffer 0 still holds the caller's histogram
      radix_clear(S, cur);
      lds_barrier();
    }
    int ib = 32 - __clz((uint32_t)(V > 1 ? V - 1 : 1));
    uint32_t ip = 0u;
    while (ib > 0) {
      const int w = ib < 8 ? ib : 8;
      ib -= w;
      const int hs = ib + w;
      const uint32_t dm = (1u << w) - 1u;
      uint32_t* h = S.hist[cur];
      visit([&](uint32_t k, uint32_t i) { hist_add(h, (i >> ib) & dm, k == tk && (i >> hs) == ip); });
      radix_clear(S, cur ^ 1);
      lds_barrier();
      radix_digit(h, nullptr, (int)dm + 1, want, false, S.bc);
      const uint32_t d = S.bc[0], below = S.bc[1], hd = S.bc[2];
      cur ^= 1;
      ip = (ip << w) | (d & dm);
      want -= below;
      if (hd == want) {
        ti = (ip << ib) | ((1u << ib) - 1u);
        break;
      }
      if (ib == 0) ti = ip;
    }
  }
  *tk_out = tk;
  *ti_out = ti;
}

__device__ __forceinline__ bool selected(uint32_t k, uint32_t i, uint32_t tk, uint32_t ti) {
  return k >= kKeyFloor && (k > tk || (k == tk && i <= ti));
}

// ---------------------------------------------------------------------------
// Fallback: exact top-`want` of the whole row by streaming it again through
// this workgroup.  Fills sel[0..n) (row order) and returns n.  The kernel
// arguments and row context come through LDS (S.fa, S.fc, written by the
// caller): the function is kept out of line so that its register pressure
// does not leak into the fast path, and handing it the by-value kernel
// argument itself would make every merge copy that argument to scratch.
// ---------------------------------------------------------------------------
template <int DT>
__device__ __attribute__((noinline)) int fallback_select(int want) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  Smem& S = *reinterpret_cast<Smem*>(smem_raw);
  uint64_t* sel = reinterpret_cast<uint64_t*>(smem_raw + kSelOff);
  const KArgs& a = S.fa;
  const Ctx& c = S.fc;
  const int tid = threadIdx.x;
  const int T = a.T;
  uint32_t nv_local = 0;
  for (int j = 0; j < T; ++j) {
    uint32_t key[kPT];
    if (tile_full(a, j * kTile))
      load_tile<DT, true>(a, c, j * kTile, S, key);
    else
      load_tile<DT, false>(a, c, j * kTile, S, key);
#pragma unroll
    for (int s = 0; s < kPT; ++s) nv_local += fold_nan(key[s]) >= kKeyFloor;
  }
  const int nv = (int)block_sum(nv_local, S.red32);
  if (want > nv) want = nv;
  if (want <= 0) return 0;
  auto visit_row = [&](auto&& f) {
    for (int j = 0; j < T; ++j) {
      uint32_t key[kPT];
      const int lo = j * kTile;
      if (tile_full(a, lo))
        load_tile<DT, true>(a, c, lo, S, key);
      else
        load_tile<DT, false>(a, c, lo, S, key);
#pragma unroll
      for (int s = 0; s < kPT; ++s) f(fold_nan(key[s]), (uint32_t)(lo + local_of_slot<DT>(tid, s)));
    }
  };
  radix_clear(S, 0);
  lds_barrier();
  uint32_t tk, ti;
  radix_select(visit_row, (uint32_t)want, (uint32_t)nv, kKeyFloor, 0xFFFFFFFFu, a.V, false, S, &tk, &ti);
  uint32_t base = 0;
  for (int j = 0; j < T; ++j) {
    uint32_t key[kPT];
    const int lo = j * kTile;
    if (tile_full(a, lo))
      load_tile<DT, true>(a, c, lo, S, key);
    else
      load_tile<DT, false>(a, c, lo, S, key);
#pragma unroll
    for (int s = 0; s < kPT; ++s) key[s] = fold_nan(key[s]);
    uint32_t cntl = 0;
#pragma unroll
    for (int s = 0; s < kPT; ++s) cntl += selected(key[s], lo + local_of_slot<DT>(tid, s), tk, ti);
    uint32_t tot;
    uint32_t off = base + block_excl_scan(cntl, S.red32, tot);
#pragma unroll
    for (int s = 0; s < kPT; ++s) {
      const uint32_t i = lo + local_of_slot<DT>(tid, s);
      if (selected(key[s], i, tk, ti)) sel[off++] = comp_of(key[s], i);
    }
    base += tot;
  }
  return (int)base;
}

// sort sel[0..n) descending (canonical order), padding to a power of two
__device__ __forceinline__ void sort_selected(uint64_t* sel, int n) {
  const int N = next_pow2(n);
  for (int r = n + (int)threadIdx.x; r < N; r += kBlock) sel[r] = 0ull;
  lds_barrier();
  lds_sort_desc(sel, N);
}

// ---------------------------------------------------------------------------
// Epilogue on the exact top-k set sel[0..n_sel): min-p filter, sort of the
// survivors, prefix sums, top-p cut (Alg. 11 order).  Leaves the sorted kept
// prefix in sel; each thread keeps the weights / inclusive sums of its chunk.
// Z_k is summed in 2^-50 fixed point so that it does not depend on the order
// in which candidates arrived.
// ---------------------------------------------------------------------------
struct Dist {
  int n_s;
  double Z_s;
  double M, tau;
  int chunk0, chunk_n;  // this thread's rows [chunk0, chunk0 + chunk_n) of sel
  double w[kEPT];       // weights of the chunk
  double incl[kEPT];    // inclusive prefix sums
};

__device__ __forceinline__ void build_dist(const KArgs& a, const Ctx& c, uint64_t Mcomp, int n_sel, Smem& S,
                                           uint64_t* sel, Dist& D) {
  const int tid = threadIdx.x;
  const int b = c.req;
  const double M = (double)float_of_key(comp_key(Mcomp));
  const double tau = (c.mode & SS_TEMP) ? (double)a.temperature[b] : 1.0;
  D.M = M;
  D.tau = tau;
  const bool minp = (c.mode & SS_MINP) && a.min_p[b] > 0.0f;
  const bool topp = (c.mode & SS_TOPP) && a.top_p[b] < 1.0f;
  const double lt = minp ? log((double)a.min_p[b]) : 0.0;

  uint64_t e[kEPT];
  uint64_t zl = 0;
  uint32_t nm_local = 0;
  uint32_t keep = 0;
#pragma unroll
  for (int m = 0; m < kEPT; ++m) {
    const int r = tid + m * kBlock;
    e[m] = 0;
    if (r < n_sel) {
      e[m] = sel[r];
      const double y = (double)float_of_key(comp_key(e[m]));
      if (topp) zl += (uint64_t)__double2ll_rn(weight_of(y, M, tau) * kFix);
      bool kp = true;
      if (minp && e[m] != Mcomp) {
        const double l = (y == M) ? 0.0 : (y - M) / tau;
        kp = l >= lt;
      }
      if (kp) {
        keep |= 1u << m;
        ++nm_local;
      }
    }
  }
  const double Zk = topp ? (double)block_sum(zl, S.red64) / kFix : 0.0;
  uint32_t n_m;
  uint32_t off = block_excl_scan(nm_local, S.red32, n_m);  // ends with a barrier: sel reads done
#pragma unroll
  for (int m = 0; m < kEPT; ++m)
    if ((keep >> m) & 1u) sel[off++] = e[m];
  const int N = next_pow2((int)n_m);
  for (int r = (int)n_m + tid; r < N; r += kBlock) sel[r] = 0ull;
  lds_barrier();
  lds_sort_desc(sel, N);

  // prefix sums over the sorted min-p prefix, chunked per thread
  const int cs = ((int)n_m + kBlock - 1) / kBlock;
  D.chunk0 = tid * cs;
  D.chunk_n = max(0, min(cs, (int)n_m - D.chunk0));
  double loc = 0.0;
  double excl_loc[kEPT];
#pragma unroll
  for (int m = 0; m < kEPT; ++m) {
    D.w[m] = 0.0;
    excl_loc[m] = 0.0;
    if (m < D.chunk_n) {
      const double y = (double)float_of_key(comp_key(sel[D.chunk0 + m]));
      D.w[m] = weight_of(y, M, tau);
      excl_loc[m] = loc;
      loc += D.w[m];
      D.incl[m] = loc;
    }
  }
  double tot;
  const double base = block_excl_scan(loc, S.redd, tot);
  uint32_t np_local = 0;
  const double thr = topp ? (double)a.top_p[b] * Zk : 0.0;
#pragma unroll
  for (int m = 0; m < kEPT; ++m) {
    if (m < D.chunk_n) {
      D.incl[m] += base;
      if (topp && base + excl_loc[m] < thr) ++np_local;
    }
  }
  int n_s = (int)n_m;
  if (topp) {
    int np = (int)block_sum(np_local, S.red32);
    if (np < 1) np = 1;
    if (np < n_s) n_s = np;
  }
  D.n_s = n_s;
  // Z_S = inclusive prefix at rank n_s - 1
  const int last = n_s - 1;
  if (last >= D.chunk0 && last < D.chunk0 + D.chunk_n) {
#pragma unroll
    for (int m = 0; m < kEPT; ++m)
      if (D.chunk0 + m == last) S.bcd[0] = D.incl[m];
  }
  lds_barrier();
  D.Z_s = S.bcd[0];
  lds_barrier();
}

// inverse CDF over the kept prefix: first rank with inclusive sum > u * Z_S
__device__ __forceinline__ int draw_rank(const Dist& D, double u, Smem& S) {
  const double target = u * D.Z_s;
  uint32_t r = 0xFFFFFFFFu;
#pragma unroll
  for (int m = 0; m < kEPT; ++m) {
    const int rr = D.chunk0 + m;
    if (m < D.chunk_n && rr < D.n_s && D.incl[m] > target && (uint32_t)rr < r) r = (uint32_t)rr;
  }
  r = block_min(r, S.red32);
  return r == 0xFFFFFFFFu ? D.n_s - 1 : (int)r;
}

// weight of sorted rank r (broadcast through LDS)
__device__ __forceinline__ double rank_weight(const Dist& D, int r, Smem& S) {
  if (r >= D.chunk0 && r < D.chunk0 + D.chunk_n) {
#pragma unroll
    for (int m = 0; m < kEPT; ++m)
      if (D.chunk0 + m == r) S.bcd[1] = D.w[m];
  }
  lds_barrier();
  const double w = S.bcd[1];
  lds_barrier();
  return w;
}

// ---------------------------------------------------------------------------
// Exact top-`want` set of a row from its unit candidates (fast path) or by
// streaming the row again (fallback).  Writes sel[0..n) unordered.
// ---------------------------------------------------------------------------
template <int DT>
__device__ __forceinline__ int select_exact(const KArgs& a, const Ctx& c, Smem& S, uint64_t* sel, int want,
                                            uint32_t tmax, uint32_t hi_key, uint32_t ovf, uint32_t n_total,
                                            int* flags) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  uint2* cnd = reinterpret_cast<uint2*>(smem_raw + kSmemFixed);  // kRPT * kBlock staging slots
  const int tid = threadIdx.x;
  const int U = a.T * kUnits;
  const uint32_t cap = (uint32_t)a.cap;
  bool fast = ovf == 0u && n_total <= (uint32_t)(kRPT * kBlock);
  // every kept candidate lies in [tmax, hi_key]: the first radix pass is
  // taken while the candidates arrive
  const Window fw = first_window(tmax, hi_key);
  uint32_t cl = 0, keepm = 0;
  uint2 e[kRPT];
  if (fast) {
    // 1. table: slot f of the row's unit-major candidate sequence -> offset
    //    of that candidate in the row's region (kept in cnd[f].x); each
    //    wavefront fills the slots of a range of units
    {
      const int G = U >= kBlock ? 1 : kBlock / U;  // threads per unit
      for (int u = tid / G; u < U; u += kBlock / G) {
        const uint32_t p = S.prefix[u];
        const uint32_t n = S.prefix[u + 1] - p;
        for (uint32_t j = (uint32_t)(tid % G); j < n; j += (uint32_t)G) cnd[p + j].x = (uint32_t)u * cap + j;
      }
      // the first radix pass below records no low-bit flags: mark every bin
      if (tid < 64) S.low[0][tid] = 0x01010101u;
    }
    lds_barrier();
    // 2. gather: every load in flight at once; slots past n_total load the
    //    region's first entry and are dropped
    const uint2* rc = a.cand + (size_t)c.row * U * cap;
    uint32_t gi[kRPT];
#pragma unroll
    for (int m = 0; m < kRPT; ++m) {
      const uint32_t f = (uint32_t)(tid + m * kBlock);
      gi[m] = f < n_total ? cnd[f].x : 0u;
    }
#pragma unroll
    for (int m = 0; m < kRPT; ++m) e[m] = rc[gi[m]];
    // 3. keep flags, count, first radix pass
    uint32_t* h = S.hist[0];
#pragma unroll
    for (int m = 0; m < kRPT; ++m) {
      const bool keep = (uint32_t)(tid + m * kBlock) < n_total && e[m].x >= tmax;
      keepm |= keep ? (1u << m) : 0u;
      cl += keep ? 1u : 0u;
      hist_add(h, (e[m].x >> fw.sh) & fw.dm, keep);
    }
  }
  // 4. compaction of the kept candidates to cnd[0, C): the scan's barriers
  //    also order every table read above before the writes below
  uint32_t C = 0;
  const uint32_t off0 = block_excl_scan(cl, S.red32, C);
  if (fast) {
    uint32_t off = off0;
#pragma unroll
    for (int m = 0; m < kRPT; ++m)
      if ((keepm >> m) & 1u) cnd[off++] = e[m];
    if (tmax == kKeyFloor) {  // every unit emitted all of its valid elements
      if ((int)C < want) want = (int)C;
    } else if ((int)C < want) {
      fast = false;  // candidates do not provably contain the top-k
    }
  }
  if (!fast) {
    *flags |= SS_FLAG_FALLBACK;
    if (tid == 0) S.fc = c;  // S.fa was written at kernel entry
    lds_barrier();
    return fallback_select<DT>(want);
  }
  // rows of kBlock compacted slots, padded with invalid entries to a multiple of 4
  const int nrow = (((int)C + kBlock - 1) / kBlock + 3) & ~3;
  for (int i = (int)C + tid; i < nrow * kBlock; i += kBlock) cnd[i] = make_uint2(0u, 0u);
  lds_barrier();
  if (want <= 0) return 0;
  auto visit_cnd = [&](auto&& f) {
    for (int r0 = 0; r0 < nrow; r0 += 4) {
      uint2 v[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = cnd[tid + (r0 + i) * kBlock];
#pragma unroll
      for (int i = 0; i < 4; ++i) f(v[i].x, v[i].y);
    }
  };
  uint32_t tk, ti;
  radix_select(visit_cnd, (uint32_t)want, C, tmax, hi_key, a.V, true, S, &tk, &ti);
  uint32_t cntl = 0;
  visit_cnd([&](uint32_t k, uint32_t i) { cntl += selected(k, i, tk, ti) ? 1u : 0u; });
  uint32_t tot;
  uint32_t off = block_excl_scan(cntl, S.red32, tot);
  visit_cnd([&](uint32_t k, uint32_t i) {
    if (selected(k, i, tk, ti)) sel[off++] = comp_of(k, i);
  });
  return (int)tot;
}

// ---------------------------------------------------------------------------
// Row merge: one workgroup per row.
// ---------------------------------------------------------------------------
template <int DT, int OP>
__device__ __forceinline__ void merge_row(const KArgs& a, const Ctx& c, Smem& S, uint64_t* sel) {
  const int tid = threadIdx.x;
  const int row = c.row, b = c.req;
  // unit records (two consecutive units per thread)
  const int U = a.T * kUnits;
  uint64_t tcomp = 0ull;
  uint32_t tthr = 0u, tovf = 0u, nl[2] = {0u, 0u};
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int u = 2 * tid + h;
    if (u < U) {
      const uint4 r4 = a.rec[(size_t)row * U + u];
      if (r4.x >= kKeyFloor) tcomp = max(tcomp, comp_of(r4.x, r4.y));
      tthr = max(tthr, r4.z);
      tovf |= r4.w > (uint32_t)a.cap ? 1u : 0u;
      nl[h] = min(r4.w, (uint32_t)a.cap);
    }
  }
  const uint64_t Mcomp = block_max(tcomp, S.red64);
  const uint32_t tmax = block_max(tthr, S.red32);
  const uint32_t ovf = block_max(tovf, S.red32);
  uint32_t n_total;
  const uint32_t pre = block_excl_scan(nl[0] + nl[1], S.red32, n_total);
  if (2 * tid < U) S.prefix[2 * tid] = pre;
  if (2 * tid + 1 < U) S.prefix[2 * tid + 1] = pre + nl[0];
  if (tid == 0) S.prefix[U] = n_total;
  radix_clear(S, 0);
  lds_barrier();

  int flags = c.kcap ? SS_FLAG_KCAP : 0;
  const bool empty = Mcomp == 0ull;
  const int argmax = empty ? -1 : (int)comp_idx(Mcomp);
  if (empty) flags = SS_FLAG_EMPTY;

  if constexpr (OP == OP_TOPK) {
    int n_sel = 0;
    if (!empty && c.k_eff > 0) {
      n_sel = select_exact<DT>(a, c, S, sel, c.k_eff, tmax, comp_key(Mcomp), ovf, n_total, &flags);
      sort_selected(sel, n_sel);
    }
    for (int r = tid; r < a.k_cap; r += kBlock) {
      const size_t o = (size_t)b * a.k_cap + r;
      if (r < n_sel) {
        a.out_val[o] = float_of_key(comp_key(sel[r]));
        a.out_idx[o] = (int32_t)comp_idx(sel[r]);
      } else {
        a.out_val[o] = -__builtin_inff();
        a.out_idx[o] = -1;
      }
    }
    if (a.flags && tid == 0) a.flags[b] = flags & SS_FLAG_FALLBACK;
    return;
  } else {
    int token = -1;
    float logprob = 0.0f;
    int accept = 0;
    const int64_t pos = a.position ? a.position[b] + c.ell : (int64_t)c.ell;
    const uint64_t seed = a.seed ? a.seed[b] : 0ull;
    bool has_draft = false;
    int dtok = -1;
    if constexpr (OP == OP_VERIFY) {
      if (c.ell < a.L) {
        dtok = a.draft_tokens[(size_t)b * a.L + c.ell];
        has_draft = dtok >= 0 && dtok < a.V;
      }
    }

    if (!empty && c.greedy) {
      token = argmax;
      if constexpr (OP == OP_VERIFY) accept = has_draft && dtok == argmax;
      if constexpr (OP == OP_PROCESS) {
        if (tid == 0) {
          RowSummary s;
          s.thr = Mcomp;
          s.Z = 1.0;
          s.M = float_of_key(comp_key(Mcomp));
          s.tau = 1.0f;
          s.argmax = argmax;
          s.kind = KIND_GREEDY;
          a.summ[row] = s;
        }
      }
      if constexpr (OP == OP_SAMPLE) {
        if (a.out_idx) {
          for (int r = tid; r < a.k_out; r += kBlock) {
            a.out_idx[(size_t)b * a.k_out + r] = r == 0 ? argmax : -1;
            a.out_prob[(size_t)b * a.k_out + r] = r == 0 ? 1.0f : 0.0f;
          }
        }
      }
    } else if (!empty) {
      const int n_sel = select_exact<DT>(a, c, S, sel, c.k_eff, tmax, comp_key(Mcomp), ovf, n_total, &flags);
      lds_barrier();
      Dist D;
      build_dist(a, c, Mcomp, n_sel, S, sel, D);
      const double u0 = uniform01(seed, (uint32_t)b, pos, 0);
      if constexpr (OP == OP_PROCESS) {
        if (tid == 0) {
          RowSummary s;
          s.thr = sel[D.n_s - 1];
          s.Z = D.Z_s;
          s.M = (float)D.M;
          s.tau = (float)D.tau;
          s.argmax = argmax;
          s.kind = KIND_DIST;
          a.summ[row] = s;
        }
      } else {
        if (OP == OP_SAMPLE || !has_draft) {
          const int r = draw_rank(D, u0, S);
          token = (int)comp_idx(sel[r]);
          const double w = rank_weight(D, r, S);
          logprob = (float)log(w / D.Z_s);
          if constexpr (OP == OP_SAMPLE) {
            if (a.out_idx) {
              for (int rr = tid; rr < a.k_out; rr += kBlock)
                a.out_idx[(size_t)b * a.k_out + rr] = rr < D.n_s ? (int32_t)comp_idx(sel[rr]) : -1;
#pragma unroll
              for (int m = 0; m < kEPT; ++m) {
                const int rr = D.chunk0 + m;
                if (m < D.chunk_n && rr < D.n_s && rr < a.k_out)
                  a.out_prob[(size_t)b * a.k_out + rr] = (float)(D.w[m] / D.Z_s);
              }
              for (int rr = D.n_s + tid; rr < a.k_out; rr += kBlock) a.out_prob[(size_t)b * a.k_out + rr] = 0.0f;
              if (D.n_s > a.k_out) flags |= SS_FLAG_OUT_TRUNC;
            }
          }
        } else {
          // verification of draft token dtok against this row's distribution
          const float* qrow = a.draft_probs + ((size_t)b * a.L + c.ell) * (size_t)a.ld_q;
          double pd_local = 0.0;
#pragma unroll
          for (int m = 0; m < kEPT; ++m) {
            const int rr = D.chunk0 + m;
            if (m < D.chunk_n && rr < D.n_s && (int)comp_idx(sel[rr]) == dtok) pd_local = D.w[m] / D.Z_s;
          }
          const double Pd = block_max(pd_local, S.redd);
          const double qd = (double)qrow[dtok];
          const double u1 = uniform01(seed, (uint32_t)b, pos, 1);
          accept = (Pd > 0.0 && u1 * qd <= Pd) ? 1 : 0;
          if (!accept) {
            // residual max(0, P - q) over the kept prefix, canonical order
            double rw[kEPT];
            double loc = 0.0;
#pragma unroll
            for (int m = 0; m < kEPT; ++m) {
              rw[m] = 0.0;
              const int rr = D.chunk0 + m;
              if (m < D.chunk_n && rr < D.n_s) {
                const double P = D.w[m] / D.Z_s;
                const double v = P - (double)qrow[comp_idx(sel[rr])];
                loc += v > 0.0 ? v : 0.0;
                rw[m] = loc;  // local inclusive prefix
              }
            }
            double Rtot;
            const double base = block_excl_scan(loc, S.redd, Rtot);
            int r;
            if (Rtot > 0.0) {
              const double target = u0 * Rtot;
              uint32_t rr_min = 0xFFFFFFFFu;
#pragma unroll
              for (int m = 0; m < kEPT; ++m) {
                const int rr = D.chunk0 + m;
                if (m < D.chunk_n && rr < D.n_s && base + rw[m] > target && (uint32_t)rr < rr_min) rr_min = rr;
              }
              rr_min = block_min(rr_min, S.red32);
              r = rr_min == 0xFFFFFFFFu ? D.n_s - 1 : (int)rr_min;
            } else {
              r = draw_rank(D, u0, S);
            }
            token = (int)comp_idx(sel[r]);
          }
        }
      }
    }

    if constexpr (OP == OP_PROCESS) {
      if (empty && tid == 0) {
        RowSummary s;
        s.thr = 0;
        s.Z = 1.0;
        s.M = 0.0f;
        s.tau = 1.0f;
        s.argmax = -1;
        s.kind = KIND_EMPTY;
        a.summ[row] = s;
      }
      if (a.flags && tid == 0) a.flags[b] = flags;
      return;
    } else if constexpr (OP == OP_SAMPLE) {
      if (tid == 0) {
        a.out_token[b] = token;
        if (a.out_logprob) a.out_logprob[b] = logprob;
        if (a.flags) a.flags[b] = flags;
      }
      if (empty && a.out_idx) {
        for (int r = tid; r < a.k_out; r += kBlock) {
          a.out_idx[(size_t)b * a.k_out + r] = -1;
          a.out_prob[(size_t)b * a.k_out + r] = 0.0f;
        }
      }
      return;
    } else {
      // publish this row's decision; the request's last row assembles
      if (tid == 0) {
        RowResult rr;
        rr.accept = accept;
        rr.emit = token;
        rr.flags = flags;
        rr.pad = 0;
        a.res[row] = rr;
      }
      __threadfence();
      __syncthreads();
      if (tid == 0) {
        const uint32_t tk = atomicAdd(&a.req_ticket[b], 1u);
        S.bc[3] = (tk == (uint32_t)a.L) ? 1u : 0u;
      }
      __syncthreads();
      if (S.bc[3] == 0u) return;
      __threadfence();
      if (tid == 0) {
        a.req_ticket[b] = 0u;
        const int L = a.L;
        int n = 0;
        int fl = 0;
        int32_t* out = a.out_tokens + (size_t)b * (L + 1);
        for (int l = 0; l <= L; ++l) out[l] = -1;
        for (int l = 0; l <= L; ++l) {
          const RowResult rr = a.res[(size_t)b * (L + 1) + l];
          fl |= rr.flags;
          if (l < L && rr.accept) {
            out[l] = a.draft_tokens[(size_t)b * L + l];
            ++n;
            continue;
          }
          out[l] = rr.emit;
          break;
        }
        a.out_nacc[b] = n;
        if (a.flags) a.flags[b] = fl;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Streaming kernel: one workgroup per (row, tile).  Tile maximum and argmax
// for every row; for truncating rows, candidate emission above a per-tile
// threshold (the q-th largest of 2048 group maxima, q = quota(k, T)).
// ---------------------------------------------------------------------------
// Largest 16-bit key prefix t with at least q of the wave's values >= t
// (binary search on the threshold; counts come from ballots, no LDS).
template <int N>
__device__ __forceinline__ uint32_t wave_threshold(const uint32_t (&v)[N], uint32_t q) {
  uint32_t prefix = 0u;
#pragma unroll 1
  for (int b = 31; b >= 16; --b) {
    const uint32_t cand = prefix | (1u << b);
    uint32_t cnt = 0u;
#pragma unroll
    for (int i = 0; i < N; ++i) cnt += (uint32_t)__popcll(__ballot(v[i] >= cand));
    if (cnt >= q) prefix = cand;
  }
  return prefix < kKeyFloor ? kKeyFloor : prefix;
}

// One tile of the streaming kernel.  After the loads everything is local to
// a wavefront: each wavefront is an emission unit with its own maximum,
// threshold and candidate region, so the tail needs no workgroup barrier.
template <int DT, bool FULL>
__device__ __forceinline__ void stream_tile(const KArgs& a, const Ctx& c, Smem& S, int row, int tile) {
  const int tid = threadIdx.x;
  const int lo = tile * kTile;
  uint32_t key[kPT];
  load_tile<DT, FULL>(a, c, lo, S, key);

  uint32_t gm[kGPT];
  auto group_maxima = [&]() {
#pragma unroll
    for (int g = 0; g < kGPT; ++g) {
      uint32_t m = key[g * kGS];
#pragma unroll
      for (int s = 1; s < kGS; ++s) m = max(m, key[g * kGS + s]);
      gm[g] = m;
    }
  };
  group_maxima();
  uint32_t tmax = gm[0];
#pragma unroll
  for (int g = 1; g < kGPT; ++g) tmax = max(tmax, gm[g]);
  if (__ballot(tmax > kKeyPosInf)) {  // a positive NaN in this wavefront: fold it to invalid
#pragma unroll
    for (int j = 0; j < kPT; ++j) key[j] = fold_nan(key[j]);
    group_maxima();
    tmax = gm[0];
#pragma unroll
    for (int g = 1; g < kGPT; ++g) tmax = max(tmax, gm[g]);
  }
  // wavefront maximum and the lowest index holding it
  const uint32_t wm = wave_max(tmax);
  uint32_t aidx = 0xFFFFFFFFu;
  if (wm >= kKeyFloor && tmax == wm) {
#pragma unroll
    for (int j = kPT - 1; j >= 0; --j)
      if (key[j] == wm) aidx = (uint32_t)(lo + local_of_slot<DT>(tid, j));
  }
  aidx = wave_min(aidx);

  const int w = wave();
  const int unit = (row * a.T + tile) * kUnits + w;
  uint32_t t = kNoEmit;
  uint32_t n = 0u;
  if (!c.greedy && c.k_eff > 0) {
    if (wm < kKeyFloor) {
      t = kKeyFloor;  // nothing valid here: everything valid (nothing) is emitted
    } else {
      const int q = quota(c.k_eff, a.T * kUnits);
      if (2 * q > kUnitGroups) {
        t = kKeyFloor;
      } else if (q <= 16) {
        const uint32_t v1[1] = {tmax};
        t = wave_threshold(v1, (uint32_t)q);
      } else {
        t = wave_threshold(gm, (uint32_t)q);
      }
      uint2* region = a.cand + (size_t)unit * a.cap;
      const uint32_t cap = (uint32_t)a.cap;
#pragma unroll
      for (int j = 0; j < kPT; ++j) {
        const bool sel = key[j] >= t;
        const uint64_t m = __ballot(sel);
        if (m) {
          if (sel) {
            const uint32_t p = n + __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                              __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
            if (p < cap) region[p] = make_uint2(key[j], (uint32_t)(lo + local_of_slot<DT>(tid, j)));
          }
          n += (uint32_t)__popcll(m);
        }
      }
    }
  }
  if (lane() == 0) a.rec[unit] = make_uint4(wm, aidx, t, n);
}

template <int DT>
__global__ __launch_bounds__(kBlock) void ss_stream_kernel(KArgs a) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  Smem& S = *reinterpret_cast<Smem*>(smem_raw);
  const int row = blockIdx.x / a.T;
  const int tile = blockIdx.x - row * a.T;
  const Ctx c = make_ctx<DT>(a, row);
  // two straight-line copies: the full-tile path keeps every load in flight
  if (tile_full(a, tile * kTile))
    stream_tile<DT, true>(a, c, S, row, tile);
  else
    stream_tile<DT, false>(a, c, S, row, tile);
}

// One workgroup per row: merge the tile records and candidates of the row.
template <int DT, int OP>
__global__ __launch_bounds__(kBlock) void ss_merge_kernel(KArgs a) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  Smem& S = *reinterpret_cast<Smem*>(smem_raw);
  uint64_t* sel = reinterpret_cast<uint64_t*>(smem_raw + kSelOff);
  if (threadIdx.x == 0) S.fa = a;  // for the out-of-line fallback
  const Ctx c = make_ctx<DT>(a, blockIdx.x);
  merge_row<DT, OP>(a, c, S, sel);
}

// ---------------------------------------------------------------------------
// Materialising pass of ss_process_logits: processed logits and final
// probabilities for every element, from the per-row summary.
// ---------------------------------------------------------------------------
template <int DT>
__global__ __launch_bounds__(kBlock) void ss_materialize_kernel(KArgs a) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  Smem& S = *reinterpret_cast<Smem*>(smem_raw);
  const int tid = threadIdx.x;
  const int row = blockIdx.x / a.T;
  const int tile = blockIdx.x - row * a.T;
  const int lo = tile * kTile;
  const Ctx c = make_ctx<DT>(a, row);
  uint32_t key[kPT];
  if (tile_full(a, lo))
    load_tile<DT, true>(a, c, lo, S, key);
  else
    load_tile<DT, false>(a, c, lo, S, key);
#pragma unroll
  for (int j = 0; j < kPT; ++j) key[j] = fold_nan(key[j]);
  const RowSummary s = a.summ[row];
  const size_t ob = (size_t)row * (size_t)a.V;
  auto emit = [&](uint32_t k, uint32_t i) {
    if (a.out_logits) a.out_logits[ob + i] = k >= kKeyFloor ? float_of_key(k) : -__builtin_inff();
    if (a.out_probs) {
      float p = 0.0f;
      if (s.kind == KIND_GREEDY) {
        p = (int)i == s.argmax ? 1.0f : 0.0f;
      } else if (s.kind == KIND_DIST && k >= kKeyFloor && comp_of(k, i) >= s.thr) {
        p = (float)(weight_of((double)float_of_key(k), (double)s.M, (double)s.tau) / s.Z);
      }
      a.out_probs[ob + i] = p;
    }
  };
#pragma unroll
  for (int j = 0; j < kPT; ++j) {
    const int l = local_of_slot<DT>(tid, j);
    if (lo + l < a.V) emit(key[j], (uint32_t)(lo + l));
  }
}

__global__ void ss_zero_kernel(uint32_t* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
struct Layout {
  int T, cap, rows;
  size_t off_ticket, off_req, off_rec, off_cand, off_res, total;
  int smem;
};

static size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

static bool make_layout(int op, int B, int V, int L, int k_max, Layout* lay) {
  if (B <= 0 || V <= 0 || V > SS_MAX_V || k_max < 1 || k_max > SS_MAX_K) return false;
  if (op == OP_VERIFY && (L < 1 || L > SS_MAX_L)) return false;
  if (op < OP_TOPK || op > OP_PROCESS) return false;
  const int rows = op == OP_VERIFY ? B * (L + 1) : B;
  const int T = (V + kTile - 1) / kTile;
  const int cap = unit_cap(k_max, T * kUnits);
  size_t o = 0;
  lay->off_ticket = o;
  o = align256(o + (size_t)rows * 4);
  lay->off_req = o;
  o = align256(o + (size_t)B * 4);
  const size_t zero_end = o;
  (void)zero_end;
  lay->off_rec = o;
  o = align256(o + (size_t)rows * T * kUnits * 16);
  lay->off_cand = o;
  o = align256(o + (size_t)rows * T * kUnits * cap * 8);
  lay->off_res = o;
  const size_t res_bytes = op == OP_VERIFY ? sizeof(RowResult) : (op == OP_PROCESS ? sizeof(RowSummary) : 0);
  o = align256(o + (size_t)rows * res_bytes);
  lay->total = o;
  lay->T = T;
  lay->cap = cap;
  lay->rows = rows;
  lay->smem = kSelOff + 8 * next_pow2(k_max);
  return true;
}

static uint32_t feature_mask(const ss_params* p) {
  uint32_t f = SS_GREEDY | SS_GRAMMAR | SS_REP | SS_FREQ | SS_PRES | SS_BIAS | SS_TEMP | SS_TOPK | SS_TOPP | SS_MINP;
  if (!p->temperature) f &= ~SS_TEMP;
  if (!p->top_k) f &= ~SS_TOPK;
  if (!p->top_p) f &= ~SS_TOPP;
  if (!p->min_p) f &= ~SS_MINP;
  if (!p->rep_penalty) f &= ~SS_REP;
  if (!p->freq_penalty) f &= ~SS_FREQ;
  if (!p->pres_penalty) f &= ~SS_PRES;
  if (!p->hist_offsets || !p->hist_ids) f &= ~(SS_REP | SS_FREQ | SS_PRES);
  if (!p->bias_offsets || !p->bias_ids || !p->bias_vals) f &= ~SS_BIAS;
  if (!p->bitmask) f &= ~SS_GRAMMAR;
  return f;
}

static void fill_params(KArgs& k, const ss_params* p) {
  k.mode = p->mode;
  k.temperature = p->temperature;
  k.top_k = p->top_k;
  k.top_p = p->top_p;
  k.min_p = p->min_p;
  k.rep = p->rep_penalty;
  k.freq = p->freq_penalty;
  k.pres = p->pres_penalty;
  k.hist_off = p->hist_offsets;
  k.hist_ids = p->hist_ids;
  k.bias_off = p->bias_offsets;
  k.bias_ids = p->bias_ids;
  k.bias_vals = p->bias_vals;
  k.bitmask = p->bitmask;
  k.mask_ld = p->bitmask_ld;
  k.seed = p->seed;
  k.position = p->position;
  k.feat = feature_mask(p);
}

static int esize(int dtype) { return dtype == SS_BF16 ? 2 : 4; }

// profiling hook (ss_set_kernel_events)
static hipEvent_t g_ev_before = nullptr, g_ev_after = nullptr;

template <int DT>
static void launch_merge(const KArgs& k, dim3 grid, dim3 block, int smem, hipStream_t st) {
  switch (k.op) {
    case OP_TOPK:
      hipLaunchKernelGGL((ss_merge_kernel<DT, OP_TOPK>), grid, block, smem, st, k);
      break;
    case OP_SAMPLE:
      hipLaunchKernelGGL((ss_merge_kernel<DT, OP_SAMPLE>), grid, block, smem, st, k);
      break;
    case OP_VERIFY:
      hipLaunchKernelGGL((ss_merge_kernel<DT, OP_VERIFY>), grid, block, smem, st, k);
      break;
    default:
      hipLaunchKernelGGL((ss_merge_kernel<DT, OP_PROCESS>), grid, block, smem, st, k);
      break;
  }
}

static ss_status launch(KArgs& k, int dtype, const Layout& lay, void* ws, hipStream_t st, bool materialize) {
  unsigned char* w = reinterpret_cast<unsigned char*>(ws);
  k.T = lay.T;
  k.cap = lay.cap;
  k.ticket = reinterpret_cast<uint32_t*>(w + lay.off_ticket);
  k.req_ticket = reinterpret_cast<uint32_t*>(w + lay.off_req);
  k.rec = reinterpret_cast<uint4*>(w + lay.off_rec);
  k.cand = reinterpret_cast<uint2*>(w + lay.off_cand);
  k.res = reinterpret_cast<RowResult*>(w + lay.off_res);
  k.summ = reinterpret_cast<RowSummary*>(w + lay.off_res);
  const dim3 grid((unsigned)(lay.rows * lay.T)), rgrid((unsigned)lay.rows), block(kBlock);
  if (g_ev_before) (void)hipEventRecord(g_ev_before, st);
  if (dtype == SS_BF16)
    hipLaunchKernelGGL(ss_stream_kernel<SS_BF16>, grid, block, kSmemStream, st, k);
  else
    hipLaunchKernelGGL(ss_stream_kernel<SS_F32>, grid, block, kSmemStream, st, k);
  if (g_ev_after) (void)hipEventRecord(g_ev_after, st);
  if (dtype == SS_BF16) {
    launch_merge<SS_BF16>(k, rgrid, block, lay.smem, st);
    if (materialize) hipLaunchKernelGGL(ss_materialize_kernel<SS_BF16>, grid, block, kSmemStream, st, k);
  } else {
    launch_merge<SS_F32>(k, rgrid, block, lay.smem, st);
    if (materialize) hipLaunchKernelGGL(ss_materialize_kernel<SS_F32>, grid, block, kSmemStream, st, k);
  }
  return hipGetLastError() == hipSuccess ? SS_OK : SS_ERR_HIP;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

static bool params_ok(const ss_params* p, int B, int V, int rows) {
  if (!p || p->B != B || p->V != V || !p->mode) return false;
  if (p->bitmask && p->bitmask_ld < (int64_t)((V + 31) / 32)) return false;
  (void)rows;
  return true;
}

}  // namespace ss

using namespace ss;

extern "C" {

size_t ss_workspace_bytes(int op, int B, int V, int L, int k_max, int dtype) {
  if (dtype != SS_F32 && dtype != SS_BF16) return 0;
  Layout lay;
  if (!make_layout(op, B, V, L, k_max, &lay)) return 0;
  return lay.total;
}

ss_status ss_workspace_init(void* ws, size_t ws_bytes, void* stream) {
  if (!ws || (ws_bytes & 3u) || !aligned16(ws)) return SS_ERR_INVALID_ARG;
  const size_t n = ws_bytes / 4;
  if (n == 0) return SS_OK;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(ss_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                     reinterpret_cast<uint32_t*>(ws), n);
  return hipGetLastError() == hipSuccess ? SS_OK : SS_ERR_HIP;
}

ss_status ss_topk(const void* x, int dtype, int B, int V, int64_t ld, const int32_t* k, int k_max,
                  float* out_val, int32_t* out_idx, int32_t* flags, void* ws, size_t ws_bytes, void* stream) {
  if (!x || !out_val || !out_idx || !ws || (dtype != SS_F32 && dtype != SS_BF16) || ld < V) return SS_ERR_INVALID_ARG;
  Layout lay;
  if (!make_layout(OP_TOPK, B, V, 0, k_max, &lay)) return SS_ERR_INVALID_ARG;
  if (ws_bytes < lay.total || !aligned16(ws)) return SS_ERR_WORKSPACE;
  KArgs a = {};
  a.x = x;
  a.ld = ld;
  a.op = OP_TOPK;
  a.B = B;
  a.rows = B;
  a.V = V;
  a.L = 0;
  a.k_cap = k_max;
  a.k_out = 0;
  a.vec_ok = aligned16(x) && ((ld * esize(dtype)) % 16 == 0);
  a.feat = SS_TOPK;
  a.top_k = k;
  a.out_val = out_val;
  a.out_idx = out_idx;
  a.flags = flags;
  return launch(a, dtype, lay, ws, (hipStream_t)stream, false);
}

ss_status ss_sample(const void* logits, int dtype, int64_t ld, const ss_params* p, int k_max, int32_t* out_token,
                    float* out_logprob, int32_t* out_idx, float* out_prob, int k_out, int32_t* flags, void* ws,
                    size_t ws_bytes, void* stream) {
  if (!logits || !p || !out_token || !ws || (dtype != SS_F32 && dtype != SS_BF16)) return SS_ERR_INVALID_ARG;
  if (k_out < 0 || (k_out > 0 && (!out_idx || !out_prob))) return SS_ERR_INVALID_ARG;
  const int B = p->B, V = p->V;
  if (ld < V || !params_ok(p, B, V, B)) return SS_ERR_INVALID_ARG;
  Layout lay;
  if (!make_layout(OP_SAMPLE, B, V, 0, k_max, &lay)) return SS_ERR_INVALID_ARG;
  if (ws_bytes < lay.total || !aligned16(ws)) return SS_ERR_WORKSPACE;
  KArgs a = {};
  a.x = logits;
  a.ld = ld;
  a.op = OP_SAMPLE;
  a.B = B;
  a.rows = B;
  a.V = V;
  a.L = 0;
  a.k_cap = k_max;
  a.k_out = k_out;
  a.vec_ok = aligned16(logits) && ((ld * esize(dtype)) % 16 == 0);
  fill_params(a, p);
  a.out_token = out_token;
  a.out_logprob = out_logprob;
  a.out_idx = k_out > 0 ? out_idx : nullptr;
  a.out_prob = k_out > 0 ? out_prob : nullptr;
  a.flags = flags;
  return launch(a, dtype, lay, ws, (hipStream_t)stream, false);
}

ss_status ss_verify(const void* target_logits, int dtype, int64_t ld_row, const float* draft_probs, int64_t ld_q,
                    const int32_t* draft_tokens, int L, const ss_params* p, int k_max, int32_t* out_tokens,
                    int32_t* out_num_accepted, int32_t* flags, void* ws, size_t ws_bytes, void* stream) {
  if (!target_logits || !p || !draft_probs || !draft_tokens || !out_tokens || !out_num_accepted || !ws)
    return SS_ERR_INVALID_ARG;
  if (dtype != SS_F32 && dtype != SS_BF16) return SS_ERR_INVALID_ARG;
  const int B = p->B, V = p->V;
  if (ld_row < V || ld_q < V || !params_ok(p, B, V, B * (L + 1))) return SS_ERR_INVALID_ARG;
  if (!p->seed || !p->position) return SS_ERR_INVALID_ARG;
  Layout lay;
  if (!make_layout(OP_VERIFY, B, V, L, k_max, &lay)) return SS_ERR_INVALID_ARG;
  if (ws_bytes < lay.total || !aligned16(ws)) return SS_ERR_WORKSPACE;
  KArgs a = {};
  a.x = target_logits;
  a.ld = ld_row;
  a.op = OP_VERIFY;
  a.B = B;
  a.rows = B * (L + 1);
  a.V = V;
  a.L = L;
  a.k_cap = k_max;
  a.k_out = 0;
  a.vec_ok = aligned16(target_logits) && ((ld_row * esize(dtype)) % 16 == 0);
  fill_params(a, p);
  a.draft_probs = draft_probs;
  a.ld_q = ld_q;
  a.draft_tokens = draft_tokens;
  a.out_tokens = out_tokens;
  a.out_nacc = out_num_accepted;
  a.flags = flags;
  return launch(a, dtype, lay, ws, (hipStream_t)stream, false);
}

ss_status ss_process_logits(const void* logits, int dtype, int64_t ld, const ss_params* p, int k_max,
                            float* out_logits, float* out_probs, int32_t* flags, void* ws, size_t ws_bytes,
                            void* stream) {
  if (!logits || !p || !ws || (dtype != SS_F32 && dtype != SS_BF16)) return SS_ERR_INVALID_ARG;
  const int B = p->B, V = p->V;
  if (ld < V || !params_ok(p, B, V, B)) return SS_ERR_INVALID_ARG;
  Layout lay;
  if (!make_layout(OP_PROCESS, B, V, 0, k_max, &lay)) return SS_ERR_INVALID_ARG;
  if (ws_bytes < lay.total || !aligned16(ws)) return SS_ERR_WORKSPACE;
  KArgs a = {};
  a.x = logits;
  a.ld = ld;
  a.op = OP_PROCESS;
  a.B = B;
  a.rows = B;
  a.V = V;
  a.L = 0;
  a.k_cap = k_max;
  a.k_out = 0;
  a.vec_ok = aligned16(logits) && ((ld * esize(dtype)) % 16 == 0);
  fill_params(a, p);
  a.out_logits = out_logits;
  a.out_probs = out_probs;
  a.flags = flags;
  return launch(a, dtype, lay, ws, (hipStream_t)stream, true);
}

ss_status ss_set_kernel_events(void* before, void* after) {
  if ((before == nullptr) != (after == nullptr)) return SS_ERR_INVALID_ARG;
  g_ev_before = reinterpret_cast<hipEvent_t>(before);
  g_ev_after = reinterpret_cast<hipEvent_t>(after);
  return SS_OK;
}

const char* ss_status_string(ss_status s) {
  switch (s) {
    case SS_OK:
      return "ok";
    case SS_ERR_INVALID_ARG:
      return "invalid argument";
    case SS_ERR_UNSUPPORTED:
      return "unsupported";
    case SS_ERR_WORKSPACE:
      return "workspace too small or misaligned";
    case SS_ERR_HIP:
      return "HIP launch error";
    default:
      return "unknown status";
  }
}

}  // extern "C"
