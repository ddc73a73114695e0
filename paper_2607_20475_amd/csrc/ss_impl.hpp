// ss_impl.hpp -- device implementation shared by the kernel translation units.
//
// Two launches per call (plus a verification assembly or a materialising
// pass for ss_verify / ss_process_logits); the grids depend only on the
// shapes, nothing synchronises with the host, so every call can be captured
// in a HIP graph.
//
// Streaming kernel.  Every wavefront owns one "unit": 2048 consecutive logits
// of one row (16-byte loads, 32 elements per lane, read exactly once).  It
// turns them into order-preserving keys (grammar allow bits applied, NaN ->
// invalid), finds a unit threshold t -- the largest 16-bit key prefix such
// that at least q group maxima of the unit reach it, q being the unit's share
// of the row's top-k plus a statistical margin -- and writes every group of
// consecutive elements whose maximum reaches t to the unit's candidate region
// (when ties at t overflow the region, the lowest-index tie groups, and the
// unit's threshold becomes the composite (t, last kept index)).  This is the
// paper's bounded candidate set of the two-stage scheme (Section 3.2), chosen
// per unit by ballots instead of a per-tile sort.  The unit stream does not
// depend on the request's penalty history or logit bias: those touch at most
// a few hundred ids per row, and extra workgroups at the front of the same
// launch build each row's patch table: the listed ids' counts and ordered
// bias sums in an LDS hash, their raw logits gathered and put through the
// Appendix C.1 prologue (repetition, frequency, presence penalty, bias; Alg. 8
// order).
//
// Merge kernel, one workgroup per row:
//   1. loads the unit records and the row's patch table (a generation-tagged
//      table in the workspace is built here instead when the lists hold more
//      distinct ids than the table does);
//   2. gathers the candidate groups, drops the raw copies of patched ids and
//      keeps the elements whose composite (key, lower index first) is at or
//      above the largest unit threshold tc, plus the patched final values at
//      or above it.  If at least k of them reach tc they provably contain the
//      row's exact top-k; otherwise (candidate overflow, skewed rows, patched
//      top tokens) an exact slow path re-reads the units that could hide a
//      top-k element (greedy rows: only the units whose threshold exceeds the
//      best unpatched candidate);
//   3. selects the exact top-k (radix select, ties -> lower index) and runs
//      the Alg. 11 epilogue: temperature weights, min-p, top-p and the token
//      draw.  Top-p and the draw are "first element in canonical order whose
//      running mass crosses a target" searches, done as radix descents with
//      2^-50 fixed-point mass histograms, so no sort is needed unless the
//      caller asks for the kept list in order.
#pragma once
#include <hip/hip_runtime.h>
#include <limits.h>
#include <stddef.h>
#include <stdint.h>

#include "ss.h"
#include "ss_device.hpp"

namespace ss {

constexpr int kPBLog = 17;                  // patched-id bitmap: 2^17 bits
constexpr int kPB = 1 << kPBLog;
constexpr int kUE = 2048;                    // elements per unit (one wavefront)
constexpr int kMaxU = SS_MAX_V / kUE;        // units per row at most (512)
constexpr int kH = 2048;                     // patch hash slots (LDS)
constexpr int kProbe = 64;                   // longest probe sequence before giving up
constexpr int kGH = 16384;                   // per-row patch table in global memory (LDS table overflow)
constexpr int kGProbe = 1024;
constexpr uint32_t kLinear = 0xFFFFFFFFu;    // patched-list count meaning "look the lists up"
constexpr int kHCopies = 2;                  // privatised radix histograms
constexpr int kRB = 9;                       // widest radix digit (bits)
constexpr int kRBins = 1 << kRB;
constexpr int kHStride = kRBins + 1;
constexpr int kGT = 4096;                    // gather table entries (LDS)
constexpr int kGS = 2048;                    // candidate groups held in registers per batch
constexpr int kEBins = 1024;                 // key bins of the sampling epilogue
constexpr int kQScan = 256;                  // sparse draft lists up to this length are scanned, longer ones sorted
constexpr uint32_t kNoEmit = 0xFFFFFFFFu;    // threshold of a unit that emits nothing
constexpr double kFix = 1125899906842624.0;  // 2^50: fixed-point scale of probability mass

enum { OP_TOPK = SS_OP_TOPK, OP_SAMPLE = SS_OP_SAMPLE, OP_VERIFY = SS_OP_VERIFY, OP_PROCESS = SS_OP_PROCESS,
       OP_LOGPROBS = SS_OP_LOGPROBS,
       OP_SAMPLE_X = 5 };  // merge only: sampling with full-row truncation or the Gumbel-max draw
// the merge instantiations that sample (the plain one carries neither extension)
constexpr bool sampling_op(int op) { return op == OP_SAMPLE || op == OP_SAMPLE_X; }
enum { KIND_EMPTY = 0, KIND_GREEDY = 1, KIND_DIST = 2 };

struct RowSummary {
  uint64_t thr;  // composite key of the last kept element
  double Z;      // sum of kept weights
  float M;       // row maximum (processed logit)
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
  int op, B, rows, V, U, L, k_cap, cap, pcap, k_out, vec_ok;
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
  const float* draft_probs;  // dense q [B, L, ld_q] (NULL when sparse)
  int64_t ld_q;
  const int32_t* dq_idx;     // sparse q: ids [B, L, kq]
  const float* dq_val;       //           probabilities [B, L, kq]
  int kq;                    // entries per draft position (0: dense q)
  const float* gum;          // sampling with the Gumbel-max draw: g = ln z per token [B, ld_g] (else NULL)
  int64_t ld_g;
  const int32_t* rmap;       // verification of a tree path: path position -> target row [B, L+1] (else NULL)
  int Lt;                    // target rows per request (L+1 without a map)
  int full;                  // sampling: full-row top-p / min-p for requests without a top-k cut
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
  uint4* rec;
  uint4* cand;
  RowResult* res;
  RowSummary* summ;
  uint2* patched;      // process: per row kGH (id, final key) pairs
  uint64_t* gtag;      // per row kGH slots: (generation << 32) | (id + 1)
  uint32_t* gcnt;      // occurrence count | has-bias bit 31
  uint32_t* gfin;      // final key
  uint32_t* npatched;  // process: per row count
  int32_t* pstat;      // per row: 0 no lists, 1 patch table in ptab, 2 more ids than the table holds
  uint32_t* ptab;      // per row 2 kH words: slot ids (-1 empty), then final keys
  int patch_wgs;       // patch-table workgroups at the front of the streaming grid
  double* usum;        // log-probabilities: per unit, sum of exp((x - unit max) / tau) over its valid logits
};

// ---------------------------------------------------------------------------
// Element layout: lane l, slot s (0..31) holds element (s / VW * 64 + l) * VW
// + s % VW of its unit; a chunk of VW consecutive elements is one 16-byte load.
// Emission groups are GE consecutive elements (two key dwords).
// ---------------------------------------------------------------------------
template <int DT>
struct DTT;
template <>
struct DTT<SS_F32> {
  static constexpr int VW = 4, NLD = 8, ES = 4, GPL = 16, GE = 2;
};
template <>
struct DTT<SS_BF16> {
  static constexpr int VW = 8, NLD = 4, ES = 2, GPL = 8, GE = 4;
};

__host__ __device__ inline int groups_per_unit(int dt) { return dt == SS_BF16 ? 512 : 1024; }

// key without the positive-NaN fold; callers fold when the maximum exceeds +inf
__device__ __forceinline__ uint32_t key_raw(uint32_t u) {
  const uint32_t s = (uint32_t)((int32_t)u >> 31);
  return (u ^ s) + (s ? 1u : 0x80000000u);
}
__device__ __forceinline__ uint32_t fold_nan(uint32_t k) { return k > kKeyPosInf ? 0u : k; }

typedef unsigned short us2 __attribute__((ext_vector_type(2)));
typedef short ss2 __attribute__((ext_vector_type(2)));
// two packed bfloat16 -> two packed 16-bit keys (the upper halves of their
// float32 keys: bf16 keys have zero low halves)
__device__ __forceinline__ uint32_t key2_bf16(uint32_t d) {
  const ss2 v = __builtin_bit_cast(ss2, d);
  const uint32_t s = __builtin_bit_cast(uint32_t, (ss2)(v >> (ss2){15, 15}));
  const uint32_t c = (s & 0x80018001u) ^ 0x80008000u;
  const us2 r = __builtin_bit_cast(us2, d ^ s) + __builtin_bit_cast(us2, c);
  return __builtin_bit_cast(uint32_t, r);
}
__device__ __forceinline__ uint32_t pkmax16(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(us2, a), __builtin_bit_cast(us2, b)));
}
__device__ __forceinline__ uint32_t hmax16(uint32_t d) { return max(d & 0xFFFFu, d >> 16); }
// positive bf16 NaN keys (above +inf = 0xFF80) -> 0 in both halves
__device__ __forceinline__ uint32_t fold_nan2(uint32_t d) {
  uint32_t lo = d & 0xFFFFu, hi = d >> 16;
  lo = lo > 0xFF80u ? 0u : lo;
  hi = hi > 0xFF80u ? 0u : hi;
  return lo | (hi << 16);
}

// float32 bit pattern of element i of a row (scalar access, any alignment)
template <int DT>
__device__ __forceinline__ uint32_t load_elem_bits(const unsigned char* xrow, int64_t i) {
  if constexpr (DT == SS_F32) {
    return reinterpret_cast<const uint32_t*>(xrow)[i];
  } else {
    return ((uint32_t)reinterpret_cast<const uint16_t*>(xrow)[i]) << 16;
  }
}

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
  float tau, top_p, min_p;  // sampling parameters (tau 1 when the TEMP bit is off)
  uint64_t seed;
  int64_t pos;              // Philox position of this row
  int dtok;                 // verification: draft token of this row (-1: none)
  bool greedy;
  bool kcap;
  bool pexact;              // the patched-id bitmap is exact (V <= kPB)
  bool full_row;            // truncation over the whole row (sampling with a.full, no top-k cut)
  int k_eff;
};

// Allow bits of a target row that a tree path maps outside the tree: none
// (zero-initialised device memory, never written).
static __device__ uint32_t g_none_allowed[SS_MAX_V / 32];

// Logits row read for verification row `row` (request b, path position
// row mod (L+1)): through the path's row map when there is one; -1 when the
// map points outside the request's Lt target rows.
__device__ __forceinline__ int64_t source_row(const KArgs& a, int row) {
  if (!a.rmap) return row;
  const int b = row / (a.L + 1);
  const int t = a.rmap[row];
  return (t >= 0 && t < a.Lt) ? (int64_t)b * a.Lt + t : -1;
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
  const int64_t srow = a.op == OP_VERIFY ? source_row(a, row) : row;
  c.xrow = reinterpret_cast<const unsigned char*>(a.x) + (size_t)(srow < 0 ? 0 : srow) * (size_t)a.ld * DTT<DT>::ES;
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
  if (srow < 0) c.mask = g_none_allowed;  // every token masked
  c.rep = (m & SS_REP) ? a.rep[b] : 1.0f;
  c.freq = (m & SS_FREQ) ? a.freq[b] : 0.0f;
  c.pres = (m & SS_PRES) ? a.pres[b] : 0.0f;
  c.tau = (m & SS_TEMP) ? a.temperature[b] : 1.0f;
  c.top_p = (m & SS_TOPP) ? a.top_p[b] : 1.0f;
  c.min_p = (m & SS_MINP) ? a.min_p[b] : 0.0f;
  c.seed = a.seed ? a.seed[b] : 0ull;
  c.pos = (a.position ? a.position[b] : 0) + c.ell;
  c.dtok = -1;
  if (a.op == OP_VERIFY && c.ell < a.L) c.dtok = a.draft_tokens[(size_t)b * a.L + c.ell];
  c.kcap = false;
  c.full_row = false;
  c.pexact = a.V <= kPB;
  if (a.op == OP_TOPK) {
    c.greedy = false;
    int k = a.top_k ? a.top_k[b] : a.k_cap;
    c.k_eff = k < 0 ? 0 : (k > a.k_cap ? a.k_cap : k);
  } else if (a.op == OP_LOGPROBS) {  // the leading k_cap tokens of rows with the bit
    c.greedy = false;
    c.k_eff = (m & SS_LOGPROBS) ? a.k_cap : 0;
  } else {
    c.greedy = (m & SS_GREEDY) || ((m & SS_TEMP) && c.tau <= 0.0f);
    const int64_t kreq = ((m & SS_TOPK) && a.top_k[b] >= 1) ? (int64_t)a.top_k[b] : (int64_t)INT_MAX;
    c.k_eff = kreq < a.k_cap ? (int)kreq : a.k_cap;
    c.kcap = !c.greedy && kreq > a.k_cap;
    c.full_row = a.full && !c.greedy && !((m & SS_TOPK) && a.top_k[b] >= 1);
    if (c.greedy) c.k_eff = 1;
  }
  return c;
}

// Candidate quota of one unit when a row's top-k is spread over U units: the
// unit keeps at least its q largest elements, q well above the expected share
// k/U (five standard deviations plus six), so that the largest unit threshold
// lies below the row's k-th value except with negligible probability.
__host__ __device__ inline int quota(int k, int U) {
  if (U <= 1 || k <= 1) return k;
  const int kt = (k + U - 1) / U;
  int s = 0;
  while (s * s < kt) ++s;
  const int q = kt + 5 * s + 6;
  return q < k ? q : k;
}

// threshold groups per lane for quota q (groups of 32/G elements); 0 when the
// quota is too large for a group threshold and the unit emits all it has
__host__ __device__ inline int thr_groups(int q, int gpl) {
  for (int G = 1; G <= gpl; G <<= 1)
    if (64 * G >= 4 * q) return G;
  return 0;
}

// capacity (groups) of one unit's candidate region
__host__ __device__ inline int unit_cap(int k_cap, int U, int dt) {
  const int gpu = groups_per_unit(dt);
  const int q = quota(k_cap, U);
  if (thr_groups(q, dt == SS_BF16 ? 8 : 16) == 0) return gpu;
  // room for twice the quota, and, when less than a whole unit, for k_cap
  // elements of one unit: a row tied at its maximum then finds its top-k
  // among the lowest-index tie groups of its first unit (the tie cut keeps
  // them)
  const int ge = dt == SS_BF16 ? 4 : 2;
  const int kg = (k_cap + ge - 1) / ge;
  int c = 2 * q + 64;
  if (kg < gpu && c < kg) c = kg;
  if ((c & 63) == 0) c += 4;  // regions not a multiple of 1 KB apart: their heads spread over the memory channels
  return c < gpu ? c : gpu;
}

// ---------------------------------------------------------------------------
// Prologue of one patched element in Appendix C.1 order, each step one
// float32 op: repetition penalty, frequency and presence penalties (count >
// 0), then the logit bias.  Grammar masking is applied by the caller.
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

// ===========================================================================
// Streaming phase: one unit per wavefront
// ===========================================================================
template <int NW>
__device__ __forceinline__ uint32_t thr_search(const uint32_t (&gm)[NW], uint32_t q, int shift) {
  // largest 16-bit prefix p with at least q of the wavefront's values >= p << shift
  // (or, once exactly q values lie at or above it, that shorter prefix).  The
  // caller guarantees q <= 64 NW, so p lies between the wavefront's smallest
  // and largest prefix: the search starts at their highest differing bit.
  uint32_t lmin = gm[0], lmax = gm[0];
#pragma unroll
  for (int i = 1; i < NW; ++i) {
    lmin = min(lmin, gm[i]);
    lmax = max(lmax, gm[i]);
  }
  const uint32_t vmin = wave_min(lmin) >> shift, vmax = wave_max_u32(lmax) >> shift;
  const uint32_t diff = vmin ^ vmax;
  if (diff == 0u) return vmin << shift;
  const int hb = 31 - __clz(diff);
  uint32_t prefix = vmax & ~((2u << hb) - 1u);
#pragma unroll 1
  for (int b = hb; b >= 0; --b) {
    const uint32_t cand = (prefix | (1u << b)) << shift;
    uint32_t cnt = 0u;
#pragma unroll
    for (int i = 0; i < NW; ++i) cnt += (uint32_t)__popcll(__ballot(gm[i] >= cand));
    if (cnt >= q) {
      prefix |= 1u << b;
      // exactly q values at or above the prefix: the lower bits cannot drop
      // any of them, and a lower threshold is still a valid one
      if (cnt == q) break;
    }
  }
  return prefix << shift;
}

// threshold over G groups per lane of the 32 keys held as bf16 pairs
template <int G>
__device__ __forceinline__ uint32_t thr_bf16(const uint32_t (&kd)[16], uint32_t q) {
  constexpr int D = 16 / G;
  uint32_t gm[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    uint32_t m = kd[g * D];
#pragma unroll
    for (int j = 1; j < D; ++j) m = pkmax16(m, kd[g * D + j]);
    gm[g] = hmax16(m);
  }
  return thr_search<G>(gm, q, 0);
}
template <int G>
__device__ __forceinline__ uint32_t thr_f32(const uint32_t (&kk)[32], uint32_t q) {
  constexpr int D = 32 / G;
  uint32_t gm[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    uint32_t m = kk[g * D];
#pragma unroll
    for (int j = 1; j < D; ++j) m = max(m, kk[g * D + j]);
    gm[g] = m;
  }
  return thr_search<G>(gm, q, 16);
}

// Ties at a unit threshold t can put more groups at or above t than the
// unit's candidate region holds.  Then every group whose maximum exceeds t is
// kept (when those alone fit) together with the lowest-index groups whose
// maximum equals t, up to the capacity: the unit still holds every element
// whose composite (key, lower index first) is at or above (t, cut), where
// cut is the last element index of the last kept tie group.  gm[g] is group
// g's maximum key; group g of a lane starts at element (g / 2 * 64 + lane) VW
// + (g % 2) GE of the unit, so index order is (g / 2, lane, g % 2).  Returns
// false (a true overflow) when the groups above t alone exceed the capacity.
template <int NG, int VW, int GE>
__device__ __forceinline__ bool tie_trim(const uint32_t (&gm)[NG], uint32_t t, uint32_t cap, uint32_t& gmask,
                                         uint32_t& cut_rel) {
  const int ln = lane();
  uint32_t gtm = 0u, eqm = 0u;
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    gtm |= (gm[g] > t ? 1u : 0u) << g;
    eqm |= (gm[g] == t ? 1u : 0u) << g;
  }
  uint32_t ngt;
  (void)wave_excl_small((uint32_t)__popc(gtm), ngt);
  if (ngt > cap) return false;
  const uint32_t rem = cap - ngt;
  uint32_t keep = 0u, base = 0u, last = 0u;
#pragma unroll
  for (int c = 0; c < NG / 2; ++c) {
    const uint32_t e2 = (eqm >> (2 * c)) & 3u;
    uint32_t tc;
    uint32_t r = base + wave_excl_small((uint32_t)__popc(e2), tc);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if ((e2 >> h) & 1u) {
        if (r < rem) {
          keep |= 1u << (2 * c + h);
          last = max(last, (uint32_t)((c * 64 + ln) * VW + h * GE + GE - 1));
        }
        ++r;
      }
    }
    base += tc;
  }
  gmask = gtm | keep;
  cut_rel = wave_max_u32(last);
  return true;
}

// Temperature of a row's log-probabilities: its own when the temperature bit
// is on, tau > 0 and the row is not greedy, else 1.
__device__ __forceinline__ float lp_tau(const KArgs& a, uint32_t mode, int b) {
  if ((mode & SS_TEMP) && !(mode & SS_GREEDY) && a.temperature[b] > 0.0f) return a.temperature[b];
  return 1.0f;
}
// One term of a unit's normaliser sum, exp((v - mu) / tau) in float32 from
// the float32 reciprocal itau; the merge recomputes it bit for bit for the
// raw copies of patched ids.
__device__ __forceinline__ float lp_term(float v, float mu, float itau) { return expf((v - mu) * itau); }
// Rows whose units add their share of the full-row normaliser: requests with
// the log-probability bit, or, in full-row sampling, stochastic requests
// without a top-k cut.
__device__ __forceinline__ bool usum_row(const KArgs& a, uint32_t mode, int b) {
  if (a.op == OP_LOGPROBS) return (mode & SS_LOGPROBS) != 0u;
  if (!a.full) return false;
  const bool greedy = (mode & SS_GREEDY) || ((mode & SS_TEMP) && a.temperature[b] <= 0.0f);
  return !greedy && !((mode & SS_TOPK) && a.top_k[b] >= 1);
}

// Streams unit `gu` (wave-uniform) and writes its record and candidate groups.
// The record is (threshold key, groups written or the count that overflowed,
// unit maximum key, last index of the tie cut or ~0u when every group at or
// above the threshold was written).
template <int DT, bool LP>
__device__ __forceinline__ void scan_unit(const KArgs& a, int gu) {
  constexpr int VW = DTT<DT>::VW, NLD = DTT<DT>::NLD, ES = DTT<DT>::ES, GPL = DTT<DT>::GPL;
  const int ln = lane();
  const int row = gu / a.U;
  const int u = gu - row * a.U;
  const int lo = u * kUE;
  const int64_t srow = a.op == OP_VERIFY ? source_row(a, row) : row;
  const int n = srow < 0 ? 0 : min(kUE, a.V - lo);  // a row outside the tree reads nothing
  const int b = a.op == OP_VERIFY ? row / (a.L + 1) : row;
  const uint32_t mode = (a.op == OP_TOPK ? SS_TOPK : (a.mode ? a.mode[b] : 0u)) & a.feat;
  const uint32_t* mask = (mode & SS_GRAMMAR) ? a.bitmask + (size_t)row * (size_t)a.mask_ld : nullptr;
  const unsigned char* xrow =
      reinterpret_cast<const unsigned char*>(a.x) + (size_t)(srow < 0 ? 0 : srow) * (size_t)a.ld * ES;

  // 1. loads: the unit's chunks, then the grammar words that cover them
  uint4 r[NLD];
  if (a.vec_ok && n == kUE) {
    const uint4* src = reinterpret_cast<const uint4*>(xrow + (size_t)lo * ES);
#pragma unroll
    for (int i = 0; i < NLD; ++i) r[i] = src[i * 64 + ln];
  } else {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int l0 = (i * 64 + ln) * VW;
      uint32_t w[4] = {0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu};  // negative NaN: invalid
#pragma unroll
      for (int e = 0; e < VW; ++e) {
        if (l0 + e < n) {
          if constexpr (DT == SS_F32) {
            w[e] = reinterpret_cast<const uint32_t*>(xrow)[lo + l0 + e];
          } else {
            const uint32_t h = reinterpret_cast<const uint16_t*>(xrow)[lo + l0 + e];
            const int q = e >> 1;
            w[q] = (e & 1) ? ((w[q] & 0x0000FFFFu) | (h << 16)) : ((w[q] & 0xFFFF0000u) | h);
          }
        }
      }
      r[i] = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
  uint32_t mw[NLD];
  if (mask) {
    const int W = (a.V + 31) >> 5;
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int wi = (lo + (i * 64 + ln) * VW) >> 5;
      mw[i] = wi < W ? mask[wi] : 0u;
    }
  }

  // 2. row parameters (scalar), read while the chunks are in flight
  int k_eff;
  if (a.op == OP_TOPK) {
    const int k = a.top_k ? a.top_k[b] : a.k_cap;
    k_eff = k < 0 ? 0 : min(k, a.k_cap);
  } else if (a.op == OP_LOGPROBS) {
    k_eff = (mode & SS_LOGPROBS) ? a.k_cap : 0;
  } else {
    const bool greedy = (mode & SS_GREEDY) || ((mode & SS_TEMP) && a.temperature[b] <= 0.0f);
    k_eff = greedy ? 1 : (((mode & SS_TOPK) && a.top_k[b] >= 1) ? min(a.top_k[b], a.k_cap) : a.k_cap);
  }

  // 3. keys, unit maximum, threshold, emission
  uint4* region = a.cand + (size_t)gu * (size_t)a.cap;
  const uint32_t cap = (uint32_t)a.cap;
  uint32_t t, wm, total, cut = 0xFFFFFFFFu;
  if constexpr (DT == SS_BF16) {
    uint32_t kd[16];
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      kd[4 * i + 0] = key2_bf16(r[i].x);
      kd[4 * i + 1] = key2_bf16(r[i].y);
      kd[4 * i + 2] = key2_bf16(r[i].z);
      kd[4 * i + 3] = key2_bf16(r[i].w);
    }
    if (mask) {
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        const uint32_t bits = mw[i] >> (((i * 64 + ln) * 8) & 31);
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const uint32_t b2 = bits >> (2 * w);
          const uint32_t m = ((b2 & 1u) ? 0x0000FFFFu : 0u) | ((b2 & 2u) ? 0xFFFF0000u : 0u);
          kd[4 * i + w] &= m;
        }
      }
    }
    uint32_t lm = kd[0];
#pragma unroll
    for (int j = 1; j < 16; ++j) lm = pkmax16(lm, kd[j]);
    uint32_t wm16 = wave_max_u32(hmax16(lm));
    if (wm16 > 0xFF80u) {  // a positive NaN in this unit: fold it to invalid
#pragma unroll
      for (int j = 0; j < 16; ++j) kd[j] = fold_nan2(kd[j]);
      lm = kd[0];
#pragma unroll
      for (int j = 1; j < 16; ++j) lm = pkmax16(lm, kd[j]);
      wm16 = wave_max_u32(hmax16(lm));
    }
    if constexpr (LP) {  // the unit's share of the full-row normaliser
      if (usum_row(a, mode, b)) {
        double sl = 0.0;
        if (wm16 >= 0x0081u) {
          const float mu = float_of_key(wm16 << 16), itau = 1.0f / lp_tau(a, mode, b);
#pragma unroll
          for (int j = 0; j < 16; ++j) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const uint32_t k16 = (kd[j] >> (16 * h)) & 0xFFFFu;
              if (k16 >= 0x0081u) sl += (double)lp_term(float_of_key(k16 << 16), mu, itau);
            }
          }
        }
        sl = wave_sum(sl);
        if (ln == 0) a.usum[gu] = sl;
      }
    }
    uint32_t t16;
    if (k_eff <= 0) {
      t16 = 0x10000u;  // above every key: nothing emitted
    } else if (wm16 < 0x0081u) {
      t16 = 0x0081u;  // nothing valid
    } else {
      const uint32_t q = (uint32_t)quota(k_eff, a.U);
      const int G = thr_groups((int)q, GPL);
      if (q <= 1) t16 = wm16;
      else if (G == 1) t16 = thr_bf16<1>(kd, q);
      else if (G == 2) t16 = thr_bf16<2>(kd, q);
      else if (G == 4) t16 = thr_bf16<4>(kd, q);
      else if (G == 8) t16 = thr_bf16<8>(kd, q);
      else t16 = 0x0081u;
      t16 = max(t16, 0x0081u);
    }
    uint32_t gmask = 0u, gm[8];
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      gm[g] = hmax16(pkmax16(kd[2 * g], kd[2 * g + 1]));
      gmask |= (gm[g] >= t16) ? (1u << g) : 0u;
    }
    uint32_t off = wave_excl_small((uint32_t)__popc(gmask), total);
    if (total > cap && t16 < 0x10000u) {
      uint32_t cr;
      if (tie_trim<8, 8, 4>(gm, t16, cap, gmask, cr)) {
        cut = (uint32_t)lo + cr;
        off = wave_excl_small((uint32_t)__popc(gmask), total);
      }
    }
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      if ((gmask >> g) & 1u) {
        const uint32_t p = off + (uint32_t)__popc(gmask & ((1u << g) - 1u));
        const uint32_t idx0 = (uint32_t)(lo + ((g >> 1) * 64 + ln) * 8 + (g & 1) * 4);
        if (p < cap) region[p] = make_uint4(idx0, kd[2 * g], kd[2 * g + 1], 0u);
      }
    }
    t = t16 >= 0x10000u ? kNoEmit : (t16 << 16);
    wm = wm16 << 16;
  } else {
    uint32_t kk[32];
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      kk[4 * i + 0] = key_raw(r[i].x);
      kk[4 * i + 1] = key_raw(r[i].y);
      kk[4 * i + 2] = key_raw(r[i].z);
      kk[4 * i + 3] = key_raw(r[i].w);
    }
    if (mask) {
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        const uint32_t bits = mw[i] >> (((i * 64 + ln) * 4) & 31);
#pragma unroll
        for (int w = 0; w < 4; ++w) kk[4 * i + w] = ((bits >> w) & 1u) ? kk[4 * i + w] : 0u;
      }
    }
    uint32_t lm = kk[0];
#pragma unroll
    for (int j = 1; j < 32; ++j) lm = max(lm, kk[j]);
    wm = wave_max_u32(lm);
    if (wm > kKeyPosInf) {
#pragma unroll
      for (int j = 0; j < 32; ++j) kk[j] = fold_nan(kk[j]);
      lm = kk[0];
#pragma unroll
      for (int j = 1; j < 32; ++j) lm = max(lm, kk[j]);
      wm = wave_max_u32(lm);
    }
    if constexpr (LP) {  // the unit's share of the full-row normaliser
      if (usum_row(a, mode, b)) {
        double sl = 0.0;
        if (wm >= kKeyFloor) {
          const float mu = float_of_key(wm), itau = 1.0f / lp_tau(a, mode, b);
#pragma unroll
          for (int j = 0; j < 32; ++j)
            if (kk[j] >= kKeyFloor) sl += (double)lp_term(float_of_key(kk[j]), mu, itau);
        }
        sl = wave_sum(sl);
        if (ln == 0) a.usum[gu] = sl;
      }
    }
    if (k_eff <= 0) {
      t = kNoEmit;
    } else if (wm < kKeyFloor) {
      t = kKeyFloor;
    } else {
      const uint32_t q = (uint32_t)quota(k_eff, a.U);
      const int G = thr_groups((int)q, GPL);
      if (q <= 1) t = wm;
      else if (G == 1) t = thr_f32<1>(kk, q);
      else if (G == 2) t = thr_f32<2>(kk, q);
      else if (G == 4) t = thr_f32<4>(kk, q);
      else if (G == 8) t = thr_f32<8>(kk, q);
      else if (G == 16) t = thr_f32<16>(kk, q);
      else t = kKeyFloor;
      t = max(t, kKeyFloor);
    }
    uint32_t gmask = 0u, gm[16];
#pragma unroll
    for (int g = 0; g < 16; ++g) {
      gm[g] = max(kk[2 * g], kk[2 * g + 1]);
      gmask |= (t != kNoEmit && gm[g] >= t) ? (1u << g) : 0u;
    }
    uint32_t off = wave_excl_small((uint32_t)__popc(gmask), total);
    if (total > cap && t != kNoEmit) {
      uint32_t cr;
      if (tie_trim<16, 4, 2>(gm, t, cap, gmask, cr)) {
        cut = (uint32_t)lo + cr;
        off = wave_excl_small((uint32_t)__popc(gmask), total);
      }
    }
#pragma unroll
    for (int g = 0; g < 16; ++g) {
      if ((gmask >> g) & 1u) {
        const uint32_t p = off + (uint32_t)__popc(gmask & ((1u << g) - 1u));
        const uint32_t idx0 = (uint32_t)(lo + ((g >> 1) * 64 + ln) * 4 + (g & 1) * 2);
        if (p < cap) region[p] = make_uint4(idx0, kk[2 * g], kk[2 * g + 1], 0u);
      }
    }
  }
  if (ln == 0) a.rec[gu] = make_uint4(t, total, wm, cut);
}

// ===========================================================================
// Merge phase
// ===========================================================================
struct MSmem {
  uint64_t r64[kWaves];
  double rd[kWaves];
  uint32_t r32[kWaves];
  uint32_t bc[8];
  uint64_t bc64[4];
  double bcd[4];
  int32_t closed[kWaves];
  uint32_t flagsw;  // bit 0: hash overflow
  uint64_t x64[2][kWaves];  // scratch of the fused reductions
  uint32_t x32[3][kWaves];
  uint32_t pbits[kPB / 32];  // bit pbit(id) set for every patched id
  int32_t hk[kH];   // patched id (or -1)
  uint32_t hf[kH];  // final key
  union {
    uint32_t gtab[kGT];  // candidate slot -> group offset in the row's regions (gather)
    struct {             // radix histograms (selection and the epilogue, after the gather)
      alignas(16) uint32_t hist[2][(kHCopies * kHStride + 3) & ~3];  // rows 16-byte aligned (tie lists are read as uint4)
      uint32_t low[2][kRBins / 4];
      uint64_t mhist[kRBins];
    };
  };
  uint32_t uoff[kMaxU + 1];
  uint32_t rmask[kMaxU / 32];  // units re-read by the slow path
};
static_assert(sizeof(uint32_t) * 2 * ((kHCopies * kHStride + 3) & ~3) + 4 * 2 * (kRBins / 4) + 8 * kRBins <=
                  sizeof(uint32_t) * kGT,
              "radix histograms share the gather table's space");
constexpr int kSmemFixed = (int)((sizeof(MSmem) + 15) & ~(size_t)15);
// the largest merge footprint (sampling ops at k_max = SS_MAX_K: pcap + kBlock
// <= 2 SS_MAX_K + 512 entries) fits gfx950's 160 KiB of LDS
static_assert(kSmemFixed + 8 * (((2 * SS_MAX_K + 128 + 255) & ~255) + kBlock) <= 160 * 1024, "merge LDS too large");
// The verification epilogue keeps a sorted copy of a sparse draft list (one
// 64-bit entry per listed id) over the patch bitmap and table, which are dead
// once the candidate pool holds the final keys.
static_assert(offsetof(MSmem, hk) == offsetof(MSmem, pbits) + sizeof(uint32_t) * (kPB / 32) &&
                  offsetof(MSmem, hf) == offsetof(MSmem, hk) + sizeof(int32_t) * kH &&
                  offsetof(MSmem, pbits) % 8 == 0 &&
                  sizeof(uint32_t) * (kPB / 32 + 2 * kH) >= sizeof(uint64_t) * SS_MAX_K,
              "sparse draft list view");
__device__ __forceinline__ uint64_t* qlist_view(MSmem& S) { return reinterpret_cast<uint64_t*>(S.pbits); }
// The key-bin sampling epilogue keeps four word tables of kEBins bins over the
// patch bitmap and its mass table over the patch table's ids (dead there too).
static_assert(4 * kEBins <= kPB / 32 && 2 * kEBins <= kH, "key-bin tables over the patch tables");

__device__ __forceinline__ uint32_t hslot(int id) { return ((uint32_t)id * 2654435761u) >> 21; }  // 11 bits
static_assert(kH == 2048, "hslot assumes 2048 slots");

// Several workgroup reductions sharing one pair of barriers.
// (max of a 64-bit value and of two 32-bit values)
__device__ __forceinline__ void block_max64_2(uint64_t& w64, uint32_t& x, uint32_t& y, MSmem& S) {
  w64 = wave_max(w64);
  x = wave_max(x);
  y = wave_max(y);
  if (lane() == 0) {
    S.x64[0][wave()] = w64;
    S.x32[0][wave()] = x;
    S.x32[1][wave()] = y;
  }
  lds_barrier();
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    w64 = max(w64, S.x64[0][w]);
    x = max(x, S.x32[0][w]);
    y = max(y, S.x32[1][w]);
  }
  lds_barrier();
}
__device__ __forceinline__ void block_max3(uint32_t& x, uint32_t& y, uint32_t& z, MSmem& S) {
  x = wave_max(x);
  y = wave_max(y);
  z = wave_max(z);
  if (lane() == 0) {
    S.x32[0][wave()] = x;
    S.x32[1][wave()] = y;
    S.x32[2][wave()] = z;
  }
  lds_barrier();
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    x = max(x, S.x32[0][w]);
    y = max(y, S.x32[1][w]);
    z = max(z, S.x32[2][w]);
  }
  lds_barrier();
}
// (max of a 64-bit value, min of a 32-bit value)
__device__ __forceinline__ void block_max_min(uint64_t& x, uint32_t& y, MSmem& S) {
  x = wave_max(x);
  y = wave_min(y);
  if (lane() == 0) {
    S.x64[0][wave()] = x;
    S.x32[0][wave()] = y;
  }
  lds_barrier();
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    x = S.x64[0][w] > x ? S.x64[0][w] : x;
    y = min(y, S.x32[0][w]);
  }
  lds_barrier();
}
// (sum, min) of 64-bit values and (sum, min) of 32-bit values; the sums are
// integer, so exact in any order
__device__ __forceinline__ void block_sum_min2(uint64_t& s64, uint64_t& m64, uint32_t& s32, uint32_t& m32, MSmem& S) {
  s64 = wave_sum(s64);
  m64 = wave_min(m64);
  s32 = wave_sum(s32);
  m32 = wave_min(m32);
  if (lane() == 0) {
    S.x64[0][wave()] = s64;
    S.x64[1][wave()] = m64;
    S.x32[0][wave()] = s32;
    S.x32[1][wave()] = m32;
  }
  lds_barrier();
  s64 = 0ull;
  s32 = 0u;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    s64 += S.x64[0][w];
    m64 = S.x64[1][w] < m64 ? S.x64[1][w] : m64;
    s32 += S.x32[0][w];
    m32 = min(m32, S.x32[1][w]);
  }
  lds_barrier();
}

// Patched-id bitmap position: the id itself when V <= kPB (the bitmap is then
// exact), else an 18-bit hash (a set bit then needs a table lookup).
__device__ __forceinline__ uint32_t pbit(int id, bool exact) {
  return exact ? (uint32_t)id : (((uint32_t)id * 0x9E3779B1u) >> (32 - kPBLog));
}
// false only when id is certainly not patched (one LDS read)
__device__ __forceinline__ bool maybe_patched(const MSmem& S, int id, bool exact) {
  const uint32_t h = pbit(id, exact);
  return (S.pbits[h >> 5] >> (h & 31)) & 1u;
}
__device__ __forceinline__ int hfind(const MSmem& S, int id) {
  uint32_t s = hslot(id);
  for (int p = 0; p < kProbe; ++p) {
    const int k = S.hk[s];
    if (k == id) return (int)s;
    if (k < 0) return -1;
    s = (s + 1) & (kH - 1);
  }
  return -1;
}
__device__ __forceinline__ bool lds_patched(const MSmem& S, int id, bool exact) {
  return maybe_patched(S, id, exact) && (exact || hfind(S, id) >= 0);
}


// ---------------------------------------------------------------------------
// Patch table of a row in global memory, used when the row's history and
// bias lists hold more distinct ids than the LDS table: open addressing over
// kGH slots.  The row's merge clears the tags before it inserts (a tag of
// generation `gen` marks a slot of this call), so nothing depends on what the
// workspace held before the call.
// ---------------------------------------------------------------------------
struct PatchG {
  uint64_t* tag;
  uint32_t* cnt;
  uint32_t* fin;
  uint32_t gen;
};
__device__ __forceinline__ uint32_t ghslot(int id) { return ((uint32_t)id * 2654435761u) >> 18; }  // 14 bits
static_assert(kGH == 16384, "ghslot assumes 16384 slots");

__device__ __forceinline__ int gfind(const PatchG& g, int id) {
  const uint64_t want = ((uint64_t)g.gen << 32) | (uint32_t)(id + 1);
  uint32_t s = ghslot(id);
  for (int p = 0; p < kGProbe; ++p) {
    const uint64_t t = __hip_atomic_load(&g.tag[s], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (t == want) return (int)s;
    if ((uint32_t)(t >> 32) != g.gen) return -1;
    s = (s + 1) & (kGH - 1);
  }
  return -1;
}
// claims a slot for id (the claiming thread zeroes its count); -1 when full
__device__ __forceinline__ int gclaim(const PatchG& g, int id) {
  const uint64_t want = ((uint64_t)g.gen << 32) | (uint32_t)(id + 1);
  uint32_t s = ghslot(id);
  for (int p = 0; p < kGProbe; ++p) {
    uint64_t t = __hip_atomic_load(&g.tag[s], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    for (;;) {
      if (t == want) return (int)s;
      if ((uint32_t)(t >> 32) == g.gen) break;  // another id of this call
      const uint64_t old = atomicCAS((unsigned long long*)&g.tag[s], (unsigned long long)t, (unsigned long long)want);
      if (old == t) {
        g.cnt[s] = 0u;
        return (int)s;
      }
      t = old;
    }
    s = (s + 1) & (kGH - 1);
  }
  return -1;
}

// linear lookups in the row's lists (last resort, any list length)
__device__ __forceinline__ bool lin_info(const Ctx& c, int id, int* count, bool* hb, float* bsum) {
  int n = 0;
  for (int h = 0; h < c.nhist; ++h) n += c.hist[h] == id;
  for (int h = 0; h < c.nextra; ++h) n += c.extra[h] == id;
  float bs = 0.0f;
  bool has = false;
  for (int e = 0; e < c.nbias; ++e)
    if (c.bias_ids[e] == id) {
      bs = bs + c.bias_vals[e];
      has = true;
    }
  *count = n;
  *hb = has;
  *bsum = bs;
  return n > 0 || has;
}
// entry e of the concatenated list (history, drafts, bias ids)
__device__ __forceinline__ int lin_entry(const Ctx& c, int e) {
  if (e < c.nhist) return c.hist[e];
  e -= c.nhist;
  if (e < c.nextra) return c.extra[e];
  return c.bias_ids[e - c.nextra];
}

// ---------------------------------------------------------------------------
// Radix selection (count based).  Histograms are privatised (kHCopies copies)
// and double-buffered: the buffer of the next pass is cleared while the
// current one fills, so one barrier separates passes.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void radix_clear(MSmem& S, int buf) {
  for (int i = threadIdx.x; i < kHCopies * kHStride; i += kBlock) S.hist[buf][i] = 0u;
  if (threadIdx.x < kRBins / 4) S.low[buf][threadIdx.x] = 0u;
}
__device__ __forceinline__ void hist_add(uint32_t* h, uint32_t bin, bool pred) {
  if (pred) atomicAdd(&h[(lane() & (kHCopies - 1)) * kHStride + bin], 1u);
}
__device__ __forceinline__ void low_mark(uint32_t* low, uint32_t bin, bool pred) {
  if (pred) reinterpret_cast<uint8_t*>(low)[bin] = 1;
}

// Digit search by wave 0 over nb <= kRBins bins.  Descending: find d with
// above(d) < want <= above(d) + h[d]; ascending: the same with the bins
// below d.  Writes (d, count before d, h[d], low flag of d) to bc[0..3]; d =
// nb if the total is below `want`.
template <int BPL>
__device__ inline void radix_digit_n(const uint32_t* h, const uint32_t* low, int nb, uint32_t want, bool descending,
                                     uint32_t* bc) {
  if (threadIdx.x < 64) {
    const int l = lane();
    uint32_t cb[BPL];
    uint32_t s = 0;
#pragma unroll
    for (int u = 0; u < BPL; ++u) {
      const int r = BPL * l + u;
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
    const uint32_t total = readlane_T(inc, 63);
    uint32_t run = inc - s;
    if (l == 0) {
      bc[0] = (uint32_t)nb;
      bc[1] = total;
      bc[2] = 0u;
      bc[3] = 1u;
    }
#pragma unroll
    for (int u = 0; u < BPL; ++u) {
      const int r = BPL * l + u;
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
__device__ __forceinline__ void radix_digit(const uint32_t* h, const uint32_t* low, int nb, uint32_t want,
                                            bool descending, uint32_t* bc) {
  if (nb <= 256)
    radix_digit_n<4>(h, low, nb, want, descending, bc);
  else
    radix_digit_n<kRBins / 64>(h, low, nb, want, descending, bc);
}

// Exact selection of the `want` largest composites (key desc, index asc)
// among the n_valid valid keys a visitor produces.  visit(f) calls f(key, idx)
// for this thread's elements.  Every valid visited key lies in [lo_key,
// hi_key]: the digit passes start just below the bits the two bounds share.
// A pass whose chosen bin holds only keys with zero bits below the digit fixes
// the boundary key at once (bf16 keys leave the low 16 bits zero).  Ties at
// the boundary key take the lowest indices (indices < V).  Returns (tk, ti):
// an element is selected iff key > tk or (key == tk and idx <= ti).
template <typename Visit>
__device__ __forceinline__ void radix_select(Visit&& visit, uint32_t want, uint32_t n_valid, uint32_t lo_key, uint32_t hi_key,
                             int V, MSmem& S, uint32_t* tk_out, uint32_t* ti_out) {
  int cur = 0;
  int sh = 32 - __clz(lo_key ^ hi_key);  // bits [0, sh) vary among the keys
  uint32_t prefix = sh >= 32 ? 0u : (hi_key >> sh);
  uint32_t tk = hi_key, ti = 0xFFFFFFFFu;
  uint32_t n_tie = n_valid;
  bool ties = true;
  radix_clear(S, 0);
  lds_barrier();
  if (want >= n_valid) {  // everything valid is selected
    tk = kKeyNegInf;
    ties = false;
    sh = 0;
  }
  while (sh > 0) {
    const int w = sh < kRB ? sh : kRB;
    sh -= w;
    const int hs = sh + w;
    const uint32_t dm = (1u << w) - 1u;
    const uint32_t lm = (1u << sh) - 1u;
    uint32_t* h = S.hist[cur];
    uint32_t* lw = S.low[cur];
    visit([&](uint32_t k, uint32_t) {
      const bool part = k >= kKeyFloor && (hs >= 32 || (k >> hs) == prefix);
      const uint32_t d = (k >> sh) & dm;
      hist_add(h, d, part);
      low_mark(lw, d, part && (k & lm) != 0u);
    });
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
    uint32_t off = block_excl_scan(cnt, S.r32, tot);
    uint32_t* tl = S.hist[cur];  // free: cleared for a next pass that does not come
    visit([&](uint32_t k, uint32_t i) {
      if (k == tk) tl[off++] = i;
    });
    lds_barrier();
    if (threadIdx.x < tot) {
      const uint32_t my = tl[threadIdx.x];
      uint32_t r = 0;
      const uint32_t tot4 = tot & ~3u;
      for (uint32_t j = 0; j < tot4; j += 4) {  // four entries per LDS read
        const uint4 q = *reinterpret_cast<const uint4*>(&tl[j]);
        r += (q.x < my ? 1u : 0u) + (q.y < my ? 1u : 0u) + (q.z < my ? 1u : 0u) + (q.w < my ? 1u : 0u);
      }
      for (uint32_t j = tot4; j < tot; ++j) r += tl[j] < my ? 1u : 0u;
      if (r == want - 1u) S.bc[4] = my;
    }
    lds_barrier();
    ti = S.bc[4];
    lds_barrier();
  } else if (ties) {
    // many ties: the `want` lowest indices by index digit passes
    int ib = 32 - __clz((uint32_t)(V > 1 ? V - 1 : 1));
    uint32_t ip = 0u;
    while (ib > 0) {
      const int w = ib < kRB ? ib : kRB;
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
// Weighted crossing search over a set held in LDS (T[0..nT), slots tid + 256 m
// with fixed-point weights Wl[i], membership bit m of `inset`): the first
// element in canonical order (key descending, index ascending) whose
// inclusive running mass is >= X (strict: > X).  Radix descent with mass
// histograms, first on the key digits (bins descending), then, inside the
// group of equal keys, on the index digits (bins ascending).  Returns the
// composite key, or 0 when the whole set's mass does not reach X.
// ---------------------------------------------------------------------------
// wave 0: first non-empty bin, in scan order, whose running mass crosses X;
// writes (bin, mass before it, its count) to bc[0], bc64[0], bc[2] and its
// low-bits flag to bc[3]; bc[0] = ~0 if none
__device__ __forceinline__ void mass_digit(MSmem& S, int nb, double X, bool strict, bool descending) {
  if (threadIdx.x < 64) {
    const int l = lane();
    constexpr int BPL = 4;  // nb <= 256
    uint64_t mb[BPL];
    uint32_t cb[BPL];
    uint64_t ms = 0;
#pragma unroll
    for (int q = 0; q < BPL; ++q) {
      const int r = BPL * l + q;
      const int bin = descending ? nb - 1 - r : r;
      mb[q] = 0;
      cb[q] = 0;
      if (r < nb) {
        mb[q] = S.mhist[bin];
#pragma unroll
        for (int cp = 0; cp < kHCopies; ++cp) cb[q] += S.hist[0][cp * kHStride + bin];
      }
      ms += mb[q];
    }
    const uint64_t inc = wave_incl_scan(ms);
    uint64_t run = inc - ms;
    // the condition is monotone over non-empty bins: the lowest lane with a
    // hit holds the first one
    int hq = -1;
    uint64_t hrun = 0;
#pragma unroll
    for (int q = 0; q < BPL; ++q) {
      const int r = BPL * l + q;
      const uint64_t nr = run + mb[q];
      const bool hit = r < nb && cb[q] > 0u && (strict ? ((double)nr > X) : ((double)nr >= X));
      if (hit && hq < 0) {
        hq = q;
        hrun = run;
      }
      run = nr;
    }
    const uint64_t hm = __ballot(hq >= 0);
    if (hm == 0ull) {
      if (l == 0) S.bc[0] = 0xFFFFFFFFu;
    } else if (l == (int)__builtin_ctzll(hm)) {
      const int bin = descending ? nb - 1 - (BPL * l + hq) : BPL * l + hq;
      S.bc[0] = (uint32_t)bin;
      S.bc64[0] = hrun;
      S.bc[2] = cb[hq];
      S.bc[3] = (S.low[0][bin >> 2] >> (8 * (bin & 3))) & 255u;
    }
  }
  lds_barrier();
}

__device__ __forceinline__ uint64_t cross_find(MSmem& S, const uint2* T, const uint64_t* Wl, int nT, uint32_t inset, double X,
                                            bool strict, uint32_t lo_key, uint32_t hi_key, int V) {
  const int tid = threadIdx.x;
  const int M = (nT + kBlock - 1) / kBlock;
  // phase 0: key digits; phase 1: index digits among keys equal to tk
  int sh = 32 - __clz(lo_key ^ hi_key);
  uint32_t prefix = sh >= 32 ? 0u : (hi_key >> sh);
  uint32_t tk = hi_key;
  int phase = sh > 0 ? 0 : 1;
  int ib = 32 - __clz((uint32_t)(V > 1 ? V - 1 : 1));
  uint32_t ip = 0u;
  uint32_t cnt_last = 0xFFFFFFFFu;
  if (phase == 1) {
    // one key value in the whole set: does its mass reach X at all?
    uint64_t ml = 0;
    for (int m = 0; m < M; ++m) {
      const int i = tid + m * kBlock;
      if (i < nT && ((inset >> m) & 1u)) ml += Wl[i];
    }
    const uint64_t mt = block_sum(ml, S.r64);
    if (!(strict ? (double)mt > X : (double)mt >= X)) return 0ull;
  }
  for (;;) {
    int w, hs, csh;
    if (phase == 0) {
      w = sh < 8 ? sh : 8;
      sh -= w;
      hs = sh + w;
      csh = sh;
    } else {
      if (ib <= 0 || cnt_last == 1u) break;
      w = ib < 8 ? ib : 8;
      ib -= w;
      hs = ib + w;
      csh = ib;
    }
    const uint32_t dm = (1u << w) - 1u;
    const uint32_t lm = (1u << csh) - 1u;
    for (int i = tid; i <= (int)dm; i += kBlock) {
      S.mhist[i] = 0ull;
#pragma unroll
      for (int cp = 0; cp < kHCopies; ++cp) S.hist[0][cp * kHStride + i] = 0u;
    }
    if (tid < 64) S.low[0][tid] = 0u;
    lds_barrier();
    for (int m0 = 0; m0 < M; m0 += 4) {
      // four entries and their weights loaded before any is used
      uint2 ev[4];
      uint64_t wv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = tid + (m0 + u) * kBlock;
        ev[u] = T[i < nT ? i : 0];
        wv[u] = Wl[i < nT ? i : 0];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
      const int m = m0 + u;
      const int i = tid + m * kBlock;
      if (m < M && i < nT && ((inset >> m) & 1u)) {
        const uint2 e = ev[u];
        bool part;
        uint32_t d;
        if (phase == 0) {
          part = hs >= 32 || (e.x >> hs) == prefix;
          d = (e.x >> csh) & dm;
        } else {
          part = e.x == tk && (hs >= 32 || (e.y >> hs) == ip);
          d = (e.y >> csh) & dm;
        }
        if (part) {
          atomicAdd(&S.mhist[d], wv[u]);
          hist_add(S.hist[0], d, true);
          low_mark(S.low[0], d, phase == 0 && (e.x & lm) != 0u);
        }
      }
      }
    }
    lds_barrier();
    mass_digit(S, (int)dm + 1, X, strict, phase == 0);
    const uint32_t d = S.bc[0];
    const uint64_t before = S.bc64[0];
    const uint32_t cnt = S.bc[2], lowd = S.bc[3];
    lds_barrier();
    if (d == 0xFFFFFFFFu) return 0ull;  // the set's mass does not reach X
    X -= (double)before;
    cnt_last = cnt;
    if (phase == 0) {
      prefix = (prefix << w) | d;
      if (sh == 0 || lowd == 0u) {  // every key in the bin equals prefix << sh
        tk = prefix << sh;
        phase = 1;
      } else if (cnt == 1u) {  // a single element: resolved below
        tk = 0u;
        break;
      }
    } else {
      ip = (ip << w) | d;
    }
  }
  // the element: the only one matching the resolved prefixes
  for (int m = 0; m < M; ++m) {
    const int i = tid + m * kBlock;
    if (i < nT && ((inset >> m) & 1u)) {
      const uint2 e = T[i];
      bool match;
      if (phase == 0) match = (e.x >> sh) == prefix;
      else match = e.x == tk && (ib >= 32 || (e.y >> ib) == ip);
      if (match) {
        S.bc[5] = e.x;
        S.bc[6] = e.y;
      }
    }
  }
  lds_barrier();
  const uint64_t r = comp_of(S.bc[5], S.bc[6]);
  lds_barrier();
  return r;
}

// final key of a patched id found by a linear lookup in the row's lists
template <int DT>
__device__ __forceinline__ uint32_t lin_final(const KArgs& a, const Ctx& c, int id) {
  int cn;
  bool hb;
  float bs;
  lin_info(c, id, &cn, &hb, &bs);
  const int Wm = (a.V + 31) >> 5;
  const bool allowed = !c.mask || ((((id >> 5) < Wm ? c.mask[id >> 5] : 0u) >> (id & 31)) & 1u);
  if (!allowed) return 0u;
  return fold_nan(penalised_key(load_elem_bits<DT>(c.xrow, id), c.mode, c.rep, c.freq, c.pres, cn, hb, bs));
}

// patch modes: 0 none, 1 LDS table, 2 global table, 3 linear lookups
template <int DT>
__device__ __forceinline__ bool is_patched(const Ctx& c, const MSmem& S, int pmode, const PatchG& g, int id) {
  if (pmode == 0) return false;
  if (pmode == 1) return lds_patched(S, id, c.pexact);
  if (pmode == 2) return gfind(g, id) >= 0;
  int cn;
  bool hb;
  float bs;
  return lin_info(c, id, &cn, &hb, &bs);
}

// ---------------------------------------------------------------------------
// Exact slow path of the merge (candidate overflow, patch-table overflow,
// skewed or heavily tied rows, patched top tokens).  It visits the row's
// candidate elements from global memory: the groups of every unit not marked
// for re-reading (located by binary search on the unit offsets), every
// element of the marked units (re-read from the logits, grammar mask
// applied) and the patched final values; raw copies of patched ids are
// skipped.  Each visit applies one element-wise operation selected by an op
// code, so a single out-of-line copy per element type serves every pass.
// ---------------------------------------------------------------------------
template <int DT>
__device__ __forceinline__ int unit_of_group(const MSmem& S, int U, uint32_t f) {
  int lo = 0, hi = U - 1;  // largest u with uoff[u] <= f
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (S.uoff[mid] <= f) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// ---------------------------------------------------------------------------
// One batch of candidate groups held in registers: PER per thread (slot
// tid + kBlock m), with their group offsets (~0u: no group).
constexpr int kGPer = kGS / kBlock;
template <int PER>
struct GBatchT {
  uint32_t go[PER];
  uint4 g[PER];
};
using GBatch = GBatchT<kGPer>;
// Groups per thread of a merge's candidate batches: six where one workgroup
// per CU suffices and large-k rows then fit one batch (bf16 sampling, fp32
// top-k), four where two workgroups must share a CU (verification, 64 + 1
// rows per CU) or where six measured slower.
template <int DT, int OP>
constexpr int gather_per() {
  return ((DT == SS_BF16 && sampling_op(OP)) || (DT == SS_F32 && OP == OP_TOPK)) ? 6 : kGPer;
}

// Slot -> group offset table of the row's candidate regions (TPU threads per
// unit), when the row's groups fit it.
__device__ __forceinline__ void gather_table(const KArgs& a, MSmem& S, int U, uint32_t NG) {
  if (NG > (uint32_t)kGT) return;
  const int tid = threadIdx.x;
  const int TPU = U >= kBlock ? 1 : kBlock / U;
  for (int x = tid; x < U * TPU; x += kBlock) {
    const int u = x / TPU, sub = x - u * TPU;
    const uint32_t o = S.uoff[u], n = S.uoff[u + 1] - o;
    for (uint32_t j = (uint32_t)sub; j < n; j += (uint32_t)TPU) S.gtab[o + j] = (uint32_t)u * a.cap + j;
  }
  lds_barrier();
}

// Issues the loads of the batch starting at group f0 (every load in flight,
// nothing waits for them here).
template <int DT, int PER>
__device__ __forceinline__ void gather_issue(const KArgs& a, const MSmem& S, int row, int U, uint32_t NG, uint32_t f0,
                                             GBatchT<PER>& gb) {
  const int tid = threadIdx.x;
  const uint4* rc = a.cand + (size_t)row * U * a.cap;
  const uint32_t nb = f0 < NG ? min((uint32_t)(PER * kBlock), NG - f0) : 0u;
  const bool table = NG <= (uint32_t)kGT;
#pragma unroll
  for (int m = 0; m < PER; ++m) {
    const uint32_t q = (uint32_t)(tid + m * kBlock);
    gb.go[m] = 0xFFFFFFFFu;
    if (q < nb) {
      if (table) {
        gb.go[m] = S.gtab[f0 + q];
      } else {
        const int u = unit_of_group<DT>(S, U, f0 + q);
        gb.go[m] = (uint32_t)u * a.cap + (f0 + q - S.uoff[u]);
      }
    }
  }
#pragma unroll
  for (int m = 0; m < PER; ++m) gb.g[m] = rc[gb.go[m] == 0xFFFFFFFFu ? 0u : gb.go[m]];
}

// ---------------------------------------------------------------------------
// Greedy rows whose emitted maxima are all patched ids with final values
// below the raw maximum (a repetition penalty on the top token): the
// processed maximum then lies below every unit threshold that the pool
// covers.  Each unit emitted every element at or above its threshold (a
// composite when ties were cut by index), so the best unpatched emitted
// element B bounds every unit whose threshold is at most B; only the units
// whose threshold exceeds B (their maximum is patched) are re-read whole.  Returns the composite of the processed maximum over the
// unpatched raw values and the patched finals (LDS patch table, when `patch`).
// Units that overflowed their candidate regions are marked for re-reading
// already, and are re-read as well.
// ---------------------------------------------------------------------------
template <int DT>
__device__ __forceinline__ uint64_t greedy_refill(const KArgs& a, const Ctx& c, MSmem& S, uint32_t NG, bool patch) {
  constexpr int GE = DTT<DT>::GE, VW = DTT<DT>::VW;
  const int tid = threadIdx.x;
  const int U = a.U;
  const bool exact = c.pexact;
  auto key_of = [](const uint4& gq, int e) -> uint32_t {
    if constexpr (DT == SS_BF16) return (((e < 2 ? gq.y : gq.z) >> (16 * (e & 1))) & 0xFFFFu) << 16;
    else return e ? gq.z : gq.y;
  };
  uint64_t best = 0ull;
  // 1. the best unpatched element among the emitted groups (the slot table
  // is rebuilt: the fast path may not have run)
  gather_table(a, S, U, NG);
  for (uint32_t f0 = 0; f0 < NG; f0 += (uint32_t)kGS) {
    GBatch gb;
    gather_issue<DT>(a, S, c.row, U, NG, f0, gb);
#pragma unroll
    for (int m = 0; m < kGPer; ++m) {
      if (gb.go[m] == 0xFFFFFFFFu) continue;
#pragma unroll
      for (int e = 0; e < GE; ++e) {
        const uint32_t k = key_of(gb.g[m], e), i = gb.g[m].x + (uint32_t)e;
        if (k >= kKeyFloor && !(patch && lds_patched(S, (int)i, exact))) best = max(best, comp_of(k, i));
      }
    }
  }
  best = block_max(best, S.r64);
  // 2. units whose maximum exceeds B
  for (int u = tid; u < U; u += kBlock) {
    const uint4 r4 = a.rec[(size_t)c.row * U + u];
    if (r4.x != kNoEmit && comp_of(r4.x, r4.w) > best) atomicOr(&S.rmask[u >> 5], 1u << (u & 31));
  }
  lds_barrier();
  // 3. every element of those units (grammar mask applied, NaN invalid)
  const int W = (a.V + 31) >> 5;
  constexpr int NCH = (kUE + kBlock * VW - 1) / (kBlock * VW);  // 16-byte chunks per thread and unit
  for (int w = 0; w < (U + 31) >> 5; ++w) {
    uint32_t mk = S.rmask[w];
    while (mk) {
      const int u = w * 32 + __builtin_ctz(mk);
      mk &= mk - 1u;
      const int lo = u * kUE;
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch) {
        if ((ch * kBlock + tid) * VW >= kUE) break;
        const int l0 = lo + (ch * kBlock + tid) * VW;
        uint32_t mw = 0xFFFFFFFFu;
        if (c.mask && l0 < a.V) mw = ((l0 >> 5) < W ? c.mask[l0 >> 5] : 0u) >> (l0 & 31);
#pragma unroll
        for (int e = 0; e < VW; ++e) {
          const int i = l0 + e;
          if (i >= a.V) break;
          uint32_t k = fold_nan(key_raw(load_elem_bits<DT>(c.xrow, i)));
          if (!((mw >> e) & 1u)) k = 0u;
          if (k >= kKeyFloor && !(patch && lds_patched(S, i, exact))) best = max(best, comp_of(k, (uint32_t)i));
        }
      }
    }
  }
  // 4. the patched finals
  for (int sl = tid; patch && sl < kH; sl += kBlock) {
    const int id = S.hk[sl];
    const uint32_t k = S.hf[sl];
    if (id >= 0 && k >= kKeyFloor) best = max(best, comp_of(k, (uint32_t)id));
  }
  return block_max(best, S.r64);
}

enum { VOP_COUNT = 0, VOP_HKEY, VOP_COUNT_EQ, VOP_LIST_EQ, VOP_HIDX, VOP_COUNT_SEL, VOP_COLLECT };
struct VOp {
  int op;
  uint32_t prefix, dm, lm, tk, ti, ip;
  int sh, hs, ib;
  uint32_t* hist;
  uint32_t* low;
  uint32_t* tl;
  uint2* pool;
};

__device__ __forceinline__ void vop_apply(const VOp& o, uint32_t k, uint32_t i, uint32_t& acc, uint32_t& off) {
  switch (o.op) {
    case VOP_COUNT:
      ++acc;
      break;
    case VOP_HKEY: {
      const bool part = o.hs >= 32 || (k >> o.hs) == o.prefix;
      const uint32_t d = (k >> o.sh) & o.dm;
      hist_add(o.hist, d, part);
      low_mark(o.low, d, part && (k & o.lm) != 0u);
      break;
    }
    case VOP_COUNT_EQ:
      acc += k == o.tk ? 1u : 0u;
      break;
    case VOP_LIST_EQ:
      if (k == o.tk) o.tl[off++] = i;
      break;
    case VOP_HIDX:
      hist_add(o.hist, (i >> o.ib) & o.dm, k == o.tk && (i >> o.hs) == o.ip);
      break;
    case VOP_COUNT_SEL:
      acc += selected(k, i, o.tk, o.ti) ? 1u : 0u;
      break;
    default:  // VOP_COLLECT
      if (selected(k, i, o.tk, o.ti)) o.pool[off++] = make_uint2(k, i);
      break;
  }
}

// visits every candidate element once; returns the op's per-thread count,
// advances *off for the list-writing ops
template <int DT>
__device__ __forceinline__ uint32_t slow_visit(const KArgs& a, const Ctx& c, const MSmem& S, uint32_t NG, int nre,
                                            int pmode, const PatchG& pg, const VOp& o, uint32_t* offp) {
  constexpr int GE = DTT<DT>::GE, VW = DTT<DT>::VW;
  const int tid = threadIdx.x;
  const int U = a.U;
  const uint4* rc = a.cand + (size_t)c.row * U * a.cap;
  uint32_t acc = 0u, off = offp ? *offp : 0u;
  // 1. groups of the units that are not re-read
  for (uint32_t f0 = 0; f0 < NG; f0 += kBlock * 4) {
    uint4 g[4];
    bool ok[4];
    size_t go[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const uint32_t fi = f0 + (uint32_t)(tid + m * kBlock);
      ok[m] = false;
      go[m] = 0;
      if (fi < NG) {
        const int u = unit_of_group<DT>(S, U, fi);
        if (!((S.rmask[u >> 5] >> (u & 31)) & 1u)) {
          ok[m] = true;
          go[m] = (size_t)u * a.cap + (fi - S.uoff[u]);
        }
      }
    }
    // unconditional loads (group 0 stands in), all in flight together
#pragma unroll
    for (int m = 0; m < 4; ++m) g[m] = rc[go[m]];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      if (!ok[m]) continue;
#pragma unroll
      for (int e = 0; e < GE; ++e) {
        uint32_t k;
        if constexpr (DT == SS_BF16) k = (((e < 2 ? g[m].y : g[m].z) >> (16 * (e & 1))) & 0xFFFFu) << 16;
        else k = e ? g[m].z : g[m].y;
        const uint32_t i = g[m].x + (uint32_t)e;
        if (k >= kKeyFloor && !is_patched<DT>(c, S, pmode, pg, (int)i)) vop_apply(o, k, i, acc, off);
      }
    }
  }
  // 2. every element of the re-read units: each thread's VW consecutive
  // elements of a unit in one 16-byte load, kRU units in flight together
  if (nre > 0) {
    const int W = (a.V + 31) >> 5;
    constexpr int kRU = 8;
    auto next_unit = [&](int from) {  // first re-read unit >= from, or U
      for (int u = from; u < U; ++u)
        if ((S.rmask[u >> 5] >> (u & 31)) & 1u) return u;
      return U;
    };
    constexpr int NCH = (kUE + kBlock * VW - 1) / (kBlock * VW);  // 16-byte chunks per thread and unit
    for (int ch = 0; ch < NCH; ++ch) {
    const int l0 = (ch * kBlock + tid) * VW;
    for (int u0 = next_unit(0); u0 < U;) {
      int uj[kRU];
      uj[0] = u0;
#pragma unroll
      for (int j = 1; j < kRU; ++j) uj[j] = uj[j - 1] < U ? next_unit(uj[j - 1] + 1) : U;
      u0 = uj[kRU - 1] < U ? next_unit(uj[kRU - 1] + 1) : U;
      uint4 r[kRU];
      uint32_t mw[kRU];
#pragma unroll
      for (int j = 0; j < kRU; ++j) {
        r[j] = make_uint4(0u, 0u, 0u, 0u);
        mw[j] = 0xFFFFFFFFu;
        const int lo = uj[j] * kUE;
        if (uj[j] < U && l0 < kUE) {
          if (a.vec_ok && lo + kUE <= a.V) {
            r[j] = *reinterpret_cast<const uint4*>(c.xrow + (size_t)(lo + l0) * DTT<DT>::ES);
          } else {
            uint32_t w4[4] = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int e = 0; e < VW; ++e) {
              const int i = lo + l0 + e;
              if (i < a.V) {
                const uint32_t bits = load_elem_bits<DT>(c.xrow, i);
                if constexpr (DT == SS_F32) w4[e] = bits;
                else w4[e >> 1] |= (bits >> 16) << (16 * (e & 1));
              }
            }
            r[j] = make_uint4(w4[0], w4[1], w4[2], w4[3]);
          }
          if (c.mask) {
            const int wi = (lo + l0) >> 5;
            mw[j] = wi < W ? (c.mask[wi] >> ((lo + l0) & 31)) : 0u;
          }
        }
      }
#pragma unroll
      for (int j = 0; j < kRU; ++j) {
        if (uj[j] >= U) continue;
        const int lo = uj[j] * kUE;
        const uint32_t w4[4] = {r[j].x, r[j].y, r[j].z, r[j].w};
#pragma unroll
        for (int e = 0; e < VW; ++e) {
          const int i = lo + l0 + e;
          if (l0 >= kUE || i >= a.V) break;
          uint32_t bits;
          if constexpr (DT == SS_F32) bits = w4[e];
          else bits = ((w4[e >> 1] >> (16 * (e & 1))) & 0xFFFFu) << 16;
          uint32_t k = fold_nan(key_raw(bits));
          if (!((mw[j] >> e) & 1u)) k = 0u;
          if (k >= kKeyFloor && !is_patched<DT>(c, S, pmode, pg, i)) vop_apply(o, k, (uint32_t)i, acc, off);
        }
      }
    }
    }
  }
  // 3. patched final values
  if (pmode == 1) {
    for (int sl = tid; sl < kH; sl += kBlock)
      if (S.hk[sl] >= 0 && S.hf[sl] >= kKeyFloor) vop_apply(o, S.hf[sl], (uint32_t)S.hk[sl], acc, off);
  } else if (pmode == 2) {
    for (int s = tid; s < kGH; s += kBlock) {
      const uint64_t t = pg.tag[s];
      if ((uint32_t)(t >> 32) == pg.gen && pg.fin[s] >= kKeyFloor) vop_apply(o, pg.fin[s], (uint32_t)t - 1u, acc, off);
    }
  } else if (pmode == 3) {
    const int ne = c.nhist + c.nextra + c.nbias;
    for (int e = tid; e < ne; e += kBlock) {
      const int id = lin_entry(c, e);
      if (id < 0 || id >= a.V) continue;
      bool first = true;
      for (int e2 = 0; e2 < e && first; ++e2) first = lin_entry(c, e2) != id;
      if (!first) continue;
      const uint32_t k = lin_final<DT>(a, c, id);
      if (k >= kKeyFloor) vop_apply(o, k, (uint32_t)id, acc, off);
    }
  }
  if (offp) *offp = off;
  return acc;
}

// Exact selection of the `want` largest composites (key desc, index asc)
// among the n_valid valid candidate elements, by the same digit passes as
// radix_select, each pass one slow_visit.
template <int DT>
__device__ __forceinline__ void slow_radix(const KArgs& a, const Ctx& c, MSmem& S, uint32_t NG, int nre, int pmode,
                                        const PatchG& pg, uint32_t want, uint32_t n_valid, uint32_t* tk_out,
                                        uint32_t* ti_out) {
  VOp o = {};
  int cur = 0;
  int sh = 32;
  uint32_t prefix = 0u;
  uint32_t tk = 0xFFFFFFFFu, ti = 0xFFFFFFFFu;
  uint32_t n_tie = n_valid;
  bool ties = true;
  radix_clear(S, 0);
  lds_barrier();
  if (want >= n_valid) {
    tk = kKeyNegInf;
    ties = false;
    sh = 0;
  }
  while (sh > 0) {
    const int w = sh < 8 ? sh : 8;
    sh -= w;
    o.op = VOP_HKEY;
    o.sh = sh;
    o.hs = sh + w;
    o.dm = (1u << w) - 1u;
    o.lm = (1u << sh) - 1u;
    o.prefix = prefix;
    o.hist = S.hist[cur];
    o.low = S.low[cur];
    slow_visit<DT>(a, c, S, NG, nre, pmode, pg, o, nullptr);
    radix_clear(S, cur ^ 1);
    lds_barrier();
    radix_digit(S.hist[cur], S.low[cur], (int)o.dm + 1, want, true, S.bc);
    const uint32_t d = S.bc[0], above = S.bc[1], hd = S.bc[2], lowd = S.bc[3];
    cur ^= 1;
    if (d > o.dm) {
      tk = kKeyNegInf;
      ti = 0xFFFFFFFFu;
      ties = false;
      break;
    }
    prefix = (prefix << w) | d;
    want -= above;
    if (hd == want) {
      tk = prefix << sh;
      ti = 0xFFFFFFFFu;
      ties = false;
      break;
    }
    if (sh == 0 || lowd == 0u) {
      tk = prefix << sh;
      n_tie = hd;
      break;
    }
  }
  if (ties && n_tie <= (uint32_t)kBlock) {
    o.op = VOP_COUNT_EQ;
    o.tk = tk;
    const uint32_t cnt = slow_visit<DT>(a, c, S, NG, nre, pmode, pg, o, nullptr);
    uint32_t tot;
    uint32_t off = block_excl_scan(cnt, S.r32, tot);
    o.op = VOP_LIST_EQ;
    o.tl = S.hist[cur];
    slow_visit<DT>(a, c, S, NG, nre, pmode, pg, o, &off);
    lds_barrier();
    if (threadIdx.x < tot) {
      const uint32_t my = o.tl[threadIdx.x];
      uint32_t r = 0;
      const uint32_t tot4 = tot & ~3u;
      for (uint32_t j = 0; j < tot4; j += 4) {  // four entries per LDS read
        const uint4 q = *reinterpret_cast<const uint4*>(&o.tl[j]);
        r += (q.x < my ? 1u : 0u) + (q.y < my ? 1u : 0u) + (q.z < my ? 1u : 0u) + (q.w < my ? 1u : 0u);
      }
      for (uint32_t j = tot4; j < tot; ++j) r += o.tl[j] < my ? 1u : 0u;
      if (r == want - 1u) S.bc[4] = my;
    }
    lds_barrier();
    ti = S.bc[4];
    lds_barrier();
  } else if (ties) {
    int ib = 32 - __clz((uint32_t)(a.V > 1 ? a.V - 1 : 1));
    uint32_t ip = 0u;
    while (ib > 0) {
      const int w = ib < 8 ? ib : 8;
      ib -= w;
      o.op = VOP_HIDX;
      o.tk = tk;
      o.ib = ib;
      o.hs = ib + w;
      o.dm = (1u << w) - 1u;
      o.ip = ip;
      o.hist = S.hist[cur];
      slow_visit<DT>(a, c, S, NG, nre, pmode, pg, o, nullptr);
      radix_clear(S, cur ^ 1);
      lds_barrier();
      radix_digit(S.hist[cur], nullptr, (int)o.dm + 1, want, false, S.bc);
      const uint32_t d = S.bc[0], below = S.bc[1], hd = S.bc[2];
      cur ^= 1;
      ip = (ip << w) | (d & o.dm);
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

// v0 = the want-th largest element among those the units emitted; every
// unit whose threshold lies above v0 (or whose candidate list overflowed)
// may hide a top-k element and is re-read whole; the exact top-k of the
// result is written to pool[0, n).
template <int DT>
__device__ __forceinline__ int slow_select(const KArgs& a, const Ctx& c, MSmem& S, uint2* pool, uint32_t NG, int pmode,
                                        const PatchG& pg, int want, uint32_t* tk_out, uint32_t* ti_out) {
  const int tid = threadIdx.x;
  const int U = a.U;
  const int row = c.row;
  uint32_t tk = 0u, ti = 0u;
  int nT = 0;
  if (want == 1 && pmode <= 1) {  // greedy rows: only the units that can hold the maximum are re-read
    const uint64_t mc = greedy_refill<DT>(a, c, S, NG, pmode == 1);
    if (tid == 0) pool[0] = make_uint2(comp_key(mc), comp_idx(mc));
    lds_barrier();
    *tk_out = comp_key(mc);
    *ti_out = comp_idx(mc);
    return mc != 0ull ? 1 : 0;
  }
  VOp o = {};
  o.op = VOP_COUNT;
  uint32_t nv = slow_visit<DT>(a, c, S, NG, 0, pmode, pg, o, nullptr);
  nv = block_sum(nv, S.r32);
  uint32_t v0 = kKeyFloor, i0 = 0xFFFFFFFFu;
  if (nv >= (uint32_t)want) slow_radix<DT>(a, c, S, NG, 0, pmode, pg, (uint32_t)want, nv, &v0, &i0);
  // units whose threshold (ties cut by index) lies above the want-th candidate
  for (int u = tid; u < U; u += kBlock) {
    const uint4 r4 = a.rec[(size_t)row * U + u];
    if (r4.x != kNoEmit && comp_of(r4.x, r4.w) > comp_of(v0, i0)) atomicOr(&S.rmask[u >> 5], 1u << (u & 31));
  }
  lds_barrier();
  int nre = 0;
  for (int w = 0; w < kMaxU / 32; ++w) nre += __popc(S.rmask[w]);
  o.op = VOP_COUNT;
  uint32_t nx = slow_visit<DT>(a, c, S, NG, nre, pmode, pg, o, nullptr);
  nx = block_sum(nx, S.r32);
  if (want > (int)nx) want = (int)nx;
  if (want > 0) {
    slow_radix<DT>(a, c, S, NG, nre, pmode, pg, (uint32_t)want, nx, &tk, &ti);
    o.op = VOP_COUNT_SEL;
    o.tk = tk;
    o.ti = ti;
    const uint32_t cl = slow_visit<DT>(a, c, S, NG, nre, pmode, pg, o, nullptr);
    uint32_t tot;
    uint32_t off = block_excl_scan(cl, S.r32, tot);
    o.op = VOP_COLLECT;
    o.pool = pool;
    slow_visit<DT>(a, c, S, NG, nre, pmode, pg, o, &off);
    nT = (int)tot;
    lds_barrier();
  }
  *tk_out = tk;
  *ti_out = ti;
  return nT;
}

// Fast-path pool: every candidate element whose composite is at or above tc
// (the largest unit threshold, ties cut by index; raw copies of
// patched ids dropped) behind the nfin patched final values at or above it
// already at pool[0, nfin), in a deterministic order (batches of groups held
// in registers, block-scan offsets).  The caller issued the first batch
// (`cur`) right after the unit records, so its loads overlap the patch
// tables' copy.
// Returns the element count (elements beyond a.pcap are counted, not stored).
template <int DT, int PER>
__device__ __forceinline__ uint32_t gather_pool(const KArgs& a, const Ctx& c, MSmem& S, uint32_t NG, bool patch,
                                                uint64_t tc, uint2* pool, uint32_t& nvalid_out, uint32_t nfin,
                                                GBatchT<PER>& cur) {
  constexpr int GE = DTT<DT>::GE;
  const int tid = threadIdx.x;
  const int U = a.U;
  const uint32_t pcap = (uint32_t)a.pcap;
  const uint32_t tck = comp_key(tc), tcut = comp_idx(tc);  // tc = (key, last index of its tie cut)
  uint32_t base = nfin;
  auto key_of = [](const uint4& gq, int e) -> uint32_t {
    if constexpr (DT == SS_BF16) return (((e < 2 ? gq.y : gq.z) >> (16 * (e & 1))) & 0xFFFFu) << 16;
    else return e ? gq.z : gq.y;
  };
  // Groups start at multiples of GE, so a group's ids share one bitmap word.
  const bool exact = a.V <= kPB;
  const uint32_t pwmax = (uint32_t)((a.V + 31) >> 5) - 1u;
  constexpr int kPer = PER;
  constexpr uint32_t kBatch = (uint32_t)(PER * kBlock);
  static_assert(kPer * GE <= 32, "selection mask is 32 bits");
  // batch f0 is processed while the loads of batch f0 + kBatch are in flight
  for (uint32_t f0 = 0; f0 < NG; f0 += kBatch) {
    GBatchT<PER> nxt;
    if (f0 + kBatch < NG) gather_issue<DT>(a, S, c.row, U, NG, f0 + kBatch, nxt);
    const uint32_t(&go)[kPer] = cur.go;
    const uint4(&g)[kPer] = cur.g;
    // patched-id bitmap words (all reads issued before any is used)
    uint32_t pw[kPer];
#pragma unroll
    for (int m = 0; m < kPer; ++m) {
      pw[m] = 0u;
      if (patch && exact) pw[m] = S.pbits[go[m] == 0xFFFFFFFFu ? 0u : min(g[m].x >> 5, pwmax)];
    }
    // selection: composite (key, index) >= tc, valid, and not the raw copy of
    // a patched id (its final value is in the pool already when it is >= tc)
    uint32_t sel = 0u;
#pragma unroll
    for (int m = 0; m < kPer; ++m) {
      const bool gv = go[m] != 0xFFFFFFFFu;
#pragma unroll
      for (int e = 0; e < GE; ++e) {
        const uint32_t k = key_of(g[m], e);
        const bool at = k > tck || (k == tck && g[m].x + (uint32_t)e <= tcut);  // composite >= tc
        sel |= ((gv && at && k >= kKeyFloor) ? 1u : 0u) << (m * GE + e);
      }
    }
    if (patch) {
      if (exact) {
#pragma unroll
        for (int m = 0; m < kPer; ++m) sel &= ~(((pw[m] >> (g[m].x & 31u)) & ((1u << GE) - 1u)) << (m * GE));
      } else {
#pragma unroll
        for (int m = 0; m < kPer; ++m) {
          const uint32_t bm = (sel >> (m * GE)) & ((1u << GE) - 1u);
          if (bm != 0u) {
#pragma unroll 1
            for (int e = 0; e < GE; ++e)
              if (((bm >> e) & 1u) && lds_patched(S, (int)(g[m].x + (uint32_t)e), false)) sel &= ~(1u << (m * GE + e));
          }
        }
      }
    }
    uint32_t tot;
    uint32_t pos = base + block_excl_scan((uint32_t)__builtin_popcount(sel), S.r32, tot);
    // every element is written: a selected one to the next pool slot, the
    // others (and those beyond pcap) to this thread's dump slot past the pool
    const uint32_t dump = pcap + (uint32_t)tid;
#pragma unroll
    for (int m = 0; m < kPer; ++m) {
#pragma unroll
      for (int e = 0; e < GE; ++e) {
        const uint32_t bit = (sel >> (m * GE + e)) & 1u;
        pool[(bit != 0u && pos < pcap) ? pos : dump] = make_uint2(key_of(g[m], e), g[m].x + (uint32_t)e);
        pos += bit;
      }
    }
    base += tot;
    cur = nxt;
  }
  nvalid_out = base;
  return base;
}

// ---------------------------------------------------------------------------
// In-place stable compaction of pool[0, n) to the elements satisfying
// pred, in rounds of 4 * kBlock: a round writes only below its own first
// unread index, so no element is overwritten before it is read.
template <typename Pred>
__device__ __forceinline__ uint32_t compact_pool(MSmem& S, uint2* pool, int n, Pred&& pred) {
  const int tid = threadIdx.x;
  uint32_t base = 0u;
  for (int r0 = 0; r0 < n; r0 += 4 * kBlock) {
    uint2 e[4];
    uint32_t sel = 0u, cnt = 0u;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const int i = r0 + tid * 4 + m;
      e[m] = i < n ? pool[i] : make_uint2(0u, 0u);
      if (i < n && pred(e[m])) {
        sel |= 1u << m;
        ++cnt;
      }
    }
    uint32_t tot;
    uint32_t off = base + block_excl_scan(cnt, S.r32, tot);  // its barriers end this round's reads
#pragma unroll
    for (int m = 0; m < 4; ++m)
      if ((sel >> m) & 1u) pool[off++] = e[m];
    base += tot;
    lds_barrier();
  }
  return base;
}


// ---------------------------------------------------------------------------
// Sampling epilogue on key bins, for bf16 rows whose pool keys span fewer than
// NB consecutive 16-bit key values (Alg. 11 order, Appendix C.2-C.3); rows
// spanning up to 512 keys take the one-bin-per-thread instantiation.
// Raw bf16 values lie on the 16-bit key grid, and elements with one key share
// one weight, so the top-k boundary, Z_k, the top-p and min-p cuts, Z_S and
// the drawn key follow from per-key counts in canonical order (keys
// descending, ties by ascending index); only the drawn element's index needs
// a pass over the pool.  Penalised or biased values (the patched finals at
// the front of the pool) may fall between grid keys: such a value is placed
// before the grid elements of its bin (it exceeds their key), and a boundary
// inside a bin holding one is resolved by walking that bin's few off-grid
// values in canonical order.  The fixed-point masses are the same integers
// the element-wise epilogue sums.  Returns false, with nothing written, when
// min-p would cut inside the maximum's own key or more than 64 patched
// finals are pooled: the element-wise epilogue then handles the row.
// ---------------------------------------------------------------------------
template <int NB>  // key bins: 512 or kEBins
__device__ __forceinline__ bool sample_binned(const Ctx& c, MSmem& S, const uint2* pool, int C, int nfin,
                                              uint32_t want, uint32_t lo16, int V, int b, int& token, float& logprob) {
  static_assert(NB <= kEBins, "bin tables sized for kEBins");
  const int tid = threadIdx.x;
  const bool minp = (c.mode & SS_MINP) && c.min_p > 0.0f;
  const bool topp = (c.mode & SS_TOPP) && c.top_p < 1.0f;
  const double lt = minp ? log((double)c.min_p) : 0.0;
  if (lt > 0.0 || nfin > 64) return false;
  const double tau = (double)c.tau;
  const double itau = 1.0 / tau;
  // the pool holds the patched finals by now: the patch tables' memory is free
  uint32_t* cnt = S.pbits;                                  // grid elements per bin (bin = key16 - lo16)
  uint32_t* minix = S.pbits + kEBins;                       // lowest index of each bin's grid elements
  uint32_t* abv = S.pbits + 2 * kEBins;                     // per position: T elements before it
  uint32_t* ocnt = S.pbits + 3 * kEBins;                    // off-grid (patched) values of each bin
  uint64_t* mbf = reinterpret_cast<uint64_t*>(S.hk);        // per position: T mass before it
  for (int i = tid; i < NB; i += kBlock) {
    cnt[i] = 0u;
    minix[i] = 0xFFFFFFFFu;
    ocnt[i] = 0u;
  }
  if (tid == 0) {
    S.bc[2] = 0u;           // last position holding elements of S
    S.bc[4] = 0xFFFFFFFFu;  // top-p crossing position
    S.bc[5] = 0xFFFFFFFFu;  // first position with a value dropped by min-p
    S.bc[6] = 0xFFFFFFFFu;  // draw position
    S.bc[7] = 0u;           // largest pool key
  }
  lds_barrier();
  uint32_t kmx = 0u;
  for (int i0 = tid; i0 < C; i0 += 4 * kBlock) {
    uint2 ee[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) ee[u] = pool[i0 + u * kBlock < C ? i0 + u * kBlock : 0];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (i0 + u * kBlock < C) {
        if ((ee[u].x & 0xFFFFu) == 0u) {
          atomicAdd(&cnt[(ee[u].x >> 16) - lo16], 1u);
          atomicMin(&minix[(ee[u].x >> 16) - lo16], ee[u].y);
        } else {
          atomicAdd(&ocnt[(ee[u].x >> 16) - lo16], 1u);
        }
        kmx = max(kmx, ee[u].x);
      }
  }
  kmx = wave_max(kmx);
  if (lane() == 0) atomicMax(&S.bc[7], kmx);
  lds_barrier();
  // positions in canonical order: position p holds bin top - p, its off-grid
  // values first (they exceed its grid key), then its grid elements; thread t
  // holds positions PP t .. PP t + PP - 1 (PP = NB / kBlock)
  const uint32_t Kmax = S.bc[7];
  const uint32_t top = (Kmax >> 16) - lo16;
  const double M = (double)float_of_key(Kmax);
  auto bin_of = [&](int pos) { return (int)top - pos; };
  auto wf_of = [&](uint32_t key) -> uint64_t {
    return (uint64_t)__double2ll_rn(weight_fast((double)float_of_key(key), M, itau) * kFix);
  };
  auto grid_key = [&](int pos) { return (lo16 + (uint32_t)bin_of(pos)) << 16; };
  auto dropped = [&](uint32_t key) {
    const double y = (double)float_of_key(key);
    const double l = (y == M) ? 0.0 : (y - M) / tau;
    return !(l >= lt);
  };
  auto off_in = [&](uint32_t k, int pos) { return (k & 0xFFFFu) != 0u && (int)((k >> 16) - lo16) == bin_of(pos); };
  // the off-grid value following composite `after` in canonical order within
  // position pos (0 when none): (key << 32) | ~index
  auto next_off = [&](int pos, uint64_t after) -> uint64_t {
    uint64_t best = 0ull;
    for (int f = 0; f < nfin; ++f) {
      const uint2 e = pool[f];
      if (off_in(e.x, pos)) {
        const uint64_t cm = comp_of(e.x, e.y);
        if (cm < after && cm > best) best = cm;
      }
    }
    return best;
  };
  // Walk the first `lim` elements of position pos (off-grid values, then grid
  // elements by index) from mass `base`: with `find`, stop at the first
  // element whose inclusive mass reaches X (exceeds it when strict).  Returns
  // the elements walked and the mass after them; *idx is the stopping
  // element's index when it is off grid, else -1 with *gj its grid rank.
  auto first_j = [&](uint64_t bp, uint64_t wp, uint32_t np, double X, bool strict) -> uint32_t {
    auto ok = [&](uint32_t j) {
      const double v = (double)(bp + (uint64_t)j * wp);
      return strict ? v > X : v >= X;
    };
    uint32_t j = 1u;
    if (wp > 0ull) {
      const double jd = (X - (double)bp) / (double)wp;
      j = jd <= 1.0 ? 1u : (jd >= (double)np ? np : (uint32_t)jd);
    }
    while (j > 1u && ok(j - 1u)) --j;
    while (j < np && !ok(j)) ++j;
    return j;
  };
  auto walk = [&](int pos, uint32_t lim, uint64_t base, bool find, double X, bool strict, uint64_t* mass_out,
                  int* idx, uint32_t* gj) -> uint32_t {
    uint64_t cum = base;
    uint32_t j = 0u;
    uint64_t after = ~0ull;
    *idx = -1;
    *gj = 0u;
    while (j < lim) {
      const uint64_t nx = next_off(pos, after);
      if (nx == 0ull) break;
      ++j;
      cum += wf_of(comp_key(nx));
      after = nx;
      if (find && (strict ? (double)cum > X : (double)cum >= X)) {
        *idx = (int)comp_idx(nx);
        *mass_out = cum;
        return j;
      }
    }
    if (j < lim) {
      const uint64_t wg = wf_of(grid_key(pos));
      const uint32_t g = find ? first_j(cum, wg, lim - j, X, strict) : lim - j;
      cum += (uint64_t)g * wg;
      j += g;
      *gj = g;
    }
    *mass_out = cum;
    return j;
  };
  constexpr int PP = NB / kBlock;  // positions per thread
  static_assert(PP >= 1 && PP * kBlock == NB, "every key bin has one position");
  uint32_t ct[PP], nn[PP], fg[PP];
  uint64_t mm[PP], wg[PP];
  bool drop[PP];
#pragma unroll
  for (int h = 0; h < PP; ++h) {
    const int pos = PP * tid + h;
    const int bn = bin_of(pos);
    const uint32_t cg = bn >= 0 ? cnt[bn] : 0u;
    uint32_t co = 0u;
    uint64_t mo = 0ull;
    if (bn >= 0 && ocnt[bn] != 0u) {
      for (int f = 0; f < nfin; ++f) {  // the few off-grid values of this bin
        const uint32_t k = pool[f].x;
        if (off_in(k, pos)) {
          ++co;
          mo += wf_of(k);
        }
      }
    }
    ct[h] = cg + co;
    fg[h] = co;
    mm[h] = mo;
    wg[h] = bn >= 0 ? wf_of(grid_key(pos)) : 0ull;
    drop[h] = minp && bn >= 0 && dropped(grid_key(pos));
  }
  uint32_t tot;
  uint32_t ctt = 0u;
#pragma unroll
  for (int h = 0; h < PP; ++h) ctt += ct[h];
  const uint32_t a0 = block_excl_scan(ctt, S.r32, tot);
  uint32_t aa[PP];
#pragma unroll
  for (int h = 0; h < PP; ++h) aa[h] = h == 0 ? a0 : aa[h - 1] + ct[h - 1];
  // T: every element of the positions above the top-k boundary, the first
  // `want` minus those above at the boundary, nothing below
#pragma unroll
  for (int h = 0; h < PP; ++h) {
    const int pos = PP * tid + h;
    nn[h] = aa[h] >= want ? 0u : min(ct[h], want - aa[h]);
    if (fg[h] == 0u || nn[h] == ct[h]) {
      mm[h] = fg[h] == 0u ? (uint64_t)nn[h] * wg[h] : mm[h] + (uint64_t)(ct[h] - fg[h]) * wg[h];
    } else if (nn[h] == 0u) {
      mm[h] = 0ull;
    } else {  // the boundary inside a mixed bin: walk its first nn elements
      uint64_t ms;
      int ix;
      uint32_t g;
      walk(pos, nn[h], 0ull, false, 0.0, false, &ms, &ix, &g);
      mm[h] = ms;
    }
  }
  uint64_t Zk;
  uint64_t mmt = 0ull;
#pragma unroll
  for (int h = 0; h < PP; ++h) mmt += mm[h];
  const uint64_t b0 = block_excl_scan(mmt, S.r64, Zk);
  uint64_t bb[PP];
#pragma unroll
  for (int h = 0; h < PP; ++h) bb[h] = h == 0 ? b0 : bb[h - 1] + mm[h - 1];
  const double Xp = (double)c.top_p * (double)Zk;
  // positions grow with the lane, so a wavefront's first hit is its lowest
  // hitting lane's; one atomic per wavefront
  uint32_t fp = 0xFFFFFFFFu, fq = 0xFFFFFFFFu;
#pragma unroll
  for (int h = PP - 1; h >= 0; --h) {
    const int pos = PP * tid + h;
    abv[pos] = aa[h];
    mbf[pos] = bb[h];
    // top-p: first position whose inclusive mass reaches p Z_k
    if (topp && nn[h] > 0u && (double)(bb[h] + mm[h]) >= Xp) fp = (uint32_t)pos;
    // min-p: first position whose grid value is dropped
    if (nn[h] > 0u && drop[h]) fq = (uint32_t)pos;
  }
  {
    const uint64_t bp = __ballot(fp != 0xFFFFFFFFu), bq = __ballot(fq != 0xFFFFFFFFu);
    if (bp != 0ull && lane() == (int)__builtin_ctzll(bp)) atomicMin(&S.bc[4], fp);
    if (bq != 0ull && lane() == (int)__builtin_ctzll(bq)) atomicMin(&S.bc[5], fq);
  }
  lds_barrier();
  auto n_at = [&](int pos) -> uint32_t {
    const uint32_t ab = abv[pos];
    return ab >= want ? 0u : min(cnt[bin_of(pos)] + ocnt[bin_of(pos)], want - ab);
  };
  // kept set S: the shorter of the two prefixes; its end (a bound on the
  // positions, and when S ends inside a position the elements of S in it)
  // and mass Z_S
  int endp = (int)top;  // no cut: S = T
  uint32_t endn = 0u;   // nonzero: S ends after this many elements of endp
  uint64_t Zs = Zk;
  const uint32_t P = S.bc[4], Q = S.bc[5];
  if (P != 0xFFFFFFFFu) {
    uint64_t ms;
    int ix;
    uint32_t g;
    const uint32_t j = walk((int)P, n_at((int)P), mbf[P], true, Xp, false, &ms, &ix, &g);
    endp = (int)P;
    endn = j;
    Zs = ms;
  }
  if (Q != 0xFFFFFFFFu && (endn == 0u || (int)Q <= endp)) {
    // min-p: position Q's grid value is dropped; only its off-grid values at
    // or above the cut (its first ones in canonical order) stay, and nothing
    // after it
    uint32_t keep = 0u;
    for (int f = 0; f < nfin; ++f) {
      const uint32_t k = pool[f].x;
      keep += (off_in(k, (int)Q) && !dropped(k)) ? 1u : 0u;
    }
    keep = min(keep, n_at((int)Q));
    if ((int)Q == endp && endn != 0u) keep = min(keep, endn);
    if (keep > 0u) {
      uint64_t ms;
      int ix;
      uint32_t g;
      walk((int)Q, keep, mbf[Q], false, 0.0, false, &ms, &ix, &g);
      Zs = ms;
      endp = (int)Q;
      endn = keep;
    } else {
      Zs = mbf[Q];
      endp = (int)Q - 1;
      endn = 0u;
    }
  }
  // draw: first element of S whose inclusive mass exceeds u Z_S; and the last
  // position holding elements of S
  const double Xd = uniform01(c.seed, (uint32_t)b, c.pos, 0) * (double)Zs;
  uint32_t fd = 0xFFFFFFFFu, ld = 0xFFFFFFFFu;
#pragma unroll
  for (int h = PP - 1; h >= 0; --h) {
    const int pos = PP * tid + h;
    if (nn[h] > 0u && pos <= endp) {
      if (ld == 0xFFFFFFFFu) ld = (uint32_t)pos;
      const uint64_t mS = (endn != 0u && pos == endp) ? Zs - bb[h] : mm[h];  // S's part of the end position
      if ((double)(bb[h] + mS) > Xd) fd = (uint32_t)pos;
    }
  }
  {
    const uint64_t bd = __ballot(fd != 0xFFFFFFFFu), bl = __ballot(ld != 0xFFFFFFFFu);
    if (bd != 0ull && lane() == (int)__builtin_ctzll(bd)) atomicMin(&S.bc[6], fd);
    if (bl != 0ull && lane() == 63 - (int)__builtin_clzll(bl)) atomicMax(&S.bc[2], ld);
  }
  lds_barrier();
  const int last = (int)S.bc[2];
  int D = (int)S.bc[6];
  if (D == (int)0xFFFFFFFF || D > last) D = last;
  const uint32_t jlim = (endn != 0u && D == endp) ? endn : n_at(D);
  const uint64_t bd = mbf[D];
  const uint32_t cd = cnt[bin_of(D)];
  const uint32_t dmin = minix[bin_of(D)];
  uint64_t md;
  int dix;
  uint32_t dgj;
  walk(D, jlim, bd, true, Xd, true, &md, &dix, &dgj);
  // every thread has read the bin tables: the index search below (or the
  // element-wise epilogue) may reuse their memory
  lds_barrier();
  if (dix < 0 && dgj == 0u) return false;  // the walk ended on no element (not expected)
  // the drawn element: an off-grid value directly, else the dgj-th lowest index
  // among the pool's grid elements of the drawn key (T holds the lowest
  // indices of the boundary key)
  uint32_t idx;
  uint32_t Kdraw;
  if (dix >= 0) {
    idx = (uint32_t)dix;
    uint32_t kd = 0u;
    for (int f = 0; f < nfin; ++f)
      if (pool[f].y == idx && off_in(pool[f].x, D)) kd = pool[f].x;
    Kdraw = kd;
  } else {
    const uint32_t Kd = grid_key(D);
    Kdraw = Kd;
    const uint32_t j = dgj;
    if (j == 1u) {
      idx = dmin;
    } else if (j == cd) {
      uint32_t r = j == 1u ? 0xFFFFFFFFu : 0u;
      for (int i = tid; i < C; i += kBlock) {
        const uint2 e = pool[i];
        if (e.x == Kd) r = j == 1u ? min(r, e.y) : max(r, e.y);
      }
      idx = j == 1u ? block_min(r, S.r32) : block_max(r, S.r32);
    } else {
      auto visit_key = [&](auto&& f) {
        for (int i = tid; i < C; i += kBlock) {
          const uint2 e = pool[i];
          if (e.x == Kd) f(e.x, e.y);
        }
      };
      uint32_t tk2, ti2;
      radix_select(visit_key, j, cd, Kd, Kd, V, S, &tk2, &ti2);
      idx = ti2;
    }
  }
  token = (int)idx;
  logprob = (float)log(weight_fast((double)float_of_key(Kdraw), M, itau) / ((double)Zs / kFix));
  return true;
}

// ---------------------------------------------------------------------------
// Row merge: the whole workgroup, after the row's last unit was written.
// ---------------------------------------------------------------------------
// This thread's share of the full-row normaliser sum_j exp((y_j - M) / tau)
// over the row's valid processed logits: the units' sums (taken by the
// streaming kernel relative to each unit's raw maximum) rescaled to M, each
// patched id's raw term (recomputed bit for bit) replaced by its final
// value's; rows whose lists exceed the LDS table recompute every element.
// The caller sums the shares over the workgroup.
template <int DT>
__device__ __forceinline__ double row_norm_part(const KArgs& a, const Ctx& c, const MSmem& S, int row, int pmode,
                                                const PatchG& pg, double M, float tauf) {
  const int U = a.U, tid = threadIdx.x;
  const float itau = 1.0f / tauf;
  const double tau = (double)tauf;
  const int Wm = (a.V + 31) >> 5;
  auto allowed = [&](int id) { return !c.mask || ((((id >> 5) < Wm ? c.mask[id >> 5] : 0u) >> (id & 31)) & 1u); };
  double z = 0.0;
  if (pmode <= 1) {
    for (int u = tid; u < U; u += kBlock) {
      const uint32_t wmu = a.rec[(size_t)row * U + u].z;
      if (wmu >= kKeyFloor) z += exp(((double)float_of_key(wmu) - M) / tau) * a.usum[(size_t)row * U + u];
    }
    for (int sl = tid; pmode == 1 && sl < kH; sl += kBlock) {
      const int id = S.hk[sl];
      if (id < 0) continue;
      uint32_t kr = fold_nan(key_raw(load_elem_bits<DT>(c.xrow, id)));  // as the unit sum counted it
      if (!allowed(id)) kr = 0u;
      if (kr >= kKeyFloor) {
        const float mu = float_of_key(a.rec[(size_t)row * U + id / kUE].z);
        z -= exp(((double)mu - M) / tau) * (double)lp_term(float_of_key(kr), mu, itau);
      }
      if (S.hf[sl] >= kKeyFloor) z += exp(((double)float_of_key(S.hf[sl]) - M) / tau);
    }
  } else {  // lists beyond the LDS table: every element's processed value
    for (int i = tid; i < a.V; i += kBlock) {
      uint32_t k = fold_nan(key_raw(load_elem_bits<DT>(c.xrow, i)));
      if (!allowed(i)) k = 0u;
      if (is_patched<DT>(c, S, pmode, pg, i)) k = pmode == 2 ? pg.fin[gfind(pg, i)] : lin_final<DT>(a, c, i);
      if (k >= kKeyFloor) z += exp(((double)float_of_key(k) - M) / tau);
    }
  }
  return z;
}

template <int DT, int OP>
__device__ __forceinline__ void merge_row(const KArgs& a, int row, MSmem& S, uint2* pool) {
  constexpr int GE = DTT<DT>::GE;
  const int tid = threadIdx.x;
  const Ctx c = make_ctx<DT>(a, row);
  const int b = c.req;
  const int U = a.U;
  const uint32_t cap = (uint32_t)a.cap;

  // the row's patch table (written by the streaming launch) is loaded up
  // front, next to the records
  const bool lists = (c.nhist + c.nextra + c.nbias) > 0;
  const int pst = lists ? a.pstat[row] : 0;
  constexpr int kTQ = kH / 4 / kBlock;  // 16-byte words per thread and table half
  uint4 tid4[kTQ], tfin4[kTQ];
  if (lists) {
    const uint4* tsrc = reinterpret_cast<const uint4*>(a.ptab + (size_t)row * 2 * kH);
#pragma unroll
    for (int m = 0; m < kTQ; ++m) {
      tid4[m] = tsrc[tid + m * kBlock];
      tfin4[m] = tsrc[kH / 4 + tid + m * kBlock];
    }
  }
  // the patched-id bitmap is cleared while the records load (the barriers of
  // the record scan order the clearing before the table's ids are set)
  const bool pexact = a.V <= kPB;
  if ((c.nhist + c.nextra + c.nbias) > 0) {
    const int pwords = pexact ? (a.V + 31) >> 5 : kPB / 32;
    for (int s = tid; s < (pwords + 3) >> 2; s += kBlock) reinterpret_cast<uint4*>(S.pbits)[s] = make_uint4(0u, 0u, 0u, 0u);
  }
  // 1. unit records: largest threshold, row maximum, candidate offsets
  uint32_t hi = 0u, ovf = 0u;
  uint64_t tc = 0ull;  // largest unit threshold as a composite (key, cut index)
  uint32_t NG = 0u;
  for (int h = 0; h * kBlock < U; ++h) {
    const int u = tid + h * kBlock;
    uint32_t cnt = 0u;
    if (u < U) {
      const uint4 r4 = a.rec[(size_t)row * U + u];
      hi = max(hi, r4.z);
      if (r4.x != kNoEmit) tc = max(tc, comp_of(r4.x, r4.w));
      if (r4.y > cap) {  // partial candidate list: the unit is re-read by the slow path
        ovf = 1u;
        atomicOr(&S.rmask[u >> 5], 1u << (u & 31));
      }
      cnt = min(r4.y, cap);
    }
    uint32_t tot;
    const uint32_t off = block_excl_scan(cnt, S.r32, tot);
    if (u < U) S.uoff[u] = NG + off;
    NG += tot;
  }
  if (tid == 0) S.uoff[U] = NG;
  if (tid == 0) S.flagsw = 0u;
  block_max64_2(tc, hi, ovf, S);
  const uint32_t tmax = comp_key(tc);  // every element at or above tc has a key >= tmax

  int flags = c.kcap ? SS_FLAG_KCAP : 0;
  const bool empty = hi < kKeyFloor;
  int want = c.k_eff;
  // the first batch of candidate groups is in flight from here on
  const bool fast = !empty && want > 0 && ovf == 0u;
  GBatchT<gather_per<DT, OP>()> cur;
  if (fast) {
    gather_table(a, S, U, NG);
    gather_issue<DT>(a, S, row, U, NG, 0u, cur);
  }

  // 2. patched ids: counts, ordered bias sums, final keys
  const bool patch = !empty && want > 0 && lists;
  int pmode = 0;
  PatchG pg;
  pg.tag = a.gtag + (size_t)row * kGH;
  pg.cnt = a.gcnt + (size_t)row * kGH;
  pg.fin = a.gfin + (size_t)row * kGH;
  pg.gen = 0u;
  const int Wm = (a.V + 31) >> 5;
  uint32_t hfmax = 0u;  // largest patched final key (LDS mode)
  uint32_t nfin0 = 0u;  // patched finals at the front of the fast-path pool
  if (patch) {
    if (pst == 1) {
      pmode = 1;
      // the table's slots as written (the hash layout is the merge's own):
      // ids and final keys, then the patched-id bitmap and the largest final
#pragma unroll
      for (int m = 0; m < kTQ; ++m) {
        reinterpret_cast<uint4*>(S.hk)[tid + m * kBlock] = tid4[m];
        reinterpret_cast<uint4*>(S.hf)[tid + m * kBlock] = tfin4[m];
      }
#pragma unroll
      for (int m = 0; m < kTQ; ++m) {
        const int ids[4] = {(int)tid4[m].x, (int)tid4[m].y, (int)tid4[m].z, (int)tid4[m].w};
        const uint32_t fk[4] = {tfin4[m].x, tfin4[m].y, tfin4[m].z, tfin4[m].w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (ids[q] < 0) continue;
          const uint32_t hb2 = pbit(ids[q], pexact);
          atomicOr(&S.pbits[hb2 >> 5], 1u << (hb2 & 31));
          hfmax = max(hfmax, fk[q]);
        }
      }
      hfmax = block_max(hfmax, S.r32);  // its barriers publish the table and the bitmap
      if (fast) {  // finals at or above tmax open the fast-path pool, in slot order
        uint32_t cnt = 0u;
#pragma unroll
        for (int m = 0; m < kTQ; ++m) {
          const int ids[4] = {(int)tid4[m].x, (int)tid4[m].y, (int)tid4[m].z, (int)tid4[m].w};
          const uint32_t fk[4] = {tfin4[m].x, tfin4[m].y, tfin4[m].z, tfin4[m].w};
#pragma unroll
          for (int q = 0; q < 4; ++q)
            cnt += (ids[q] >= 0 && comp_of(fk[q], (uint32_t)ids[q]) >= tc && fk[q] >= kKeyFloor) ? 1u : 0u;
        }
        uint32_t off = block_excl_scan(cnt, S.r32, nfin0);
#pragma unroll
        for (int m = 0; m < kTQ; ++m) {
          const int ids[4] = {(int)tid4[m].x, (int)tid4[m].y, (int)tid4[m].z, (int)tid4[m].w};
          const uint32_t fk[4] = {tfin4[m].x, tfin4[m].y, tfin4[m].z, tfin4[m].w};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if (ids[q] >= 0 && comp_of(fk[q], (uint32_t)ids[q]) >= tc && fk[q] >= kKeyFloor) {
              if (off < (uint32_t)a.pcap) pool[off] = make_uint2(fk[q], (uint32_t)ids[q]);
              ++off;
            }
          }
        }
      }
    } else {
      // more distinct ids than the LDS table holds (status 2): the row's table in global
      // memory, cleared first (its contents before the call are unspecified)
      for (int sl = tid; sl < kGH / 2; sl += kBlock) reinterpret_cast<uint4*>(pg.tag)[sl] = make_uint4(0u, 0u, 0u, 0u);
      pg.gen = 1u;
      __threadfence();
      __syncthreads();
      const int ne = c.nhist + c.nextra + c.nbias;
      bool full = false;
      for (int e = tid; e < ne; e += kBlock) {
        const int id = lin_entry(c, e);
        if (id >= 0 && id < a.V && gclaim(pg, id) < 0) full = true;
      }
      if (full) S.flagsw = 3u;
      __threadfence();
      __syncthreads();
      if (S.flagsw == 3u) {
        pmode = 3;
      } else {
        pmode = 2;
        for (int e = tid; e < ne; e += kBlock) {
          const int id = lin_entry(c, e);
          if (id < 0 || id >= a.V) continue;
          const int sl = gfind(pg, id);
          if (e < c.nhist + c.nextra) atomicAdd(&pg.cnt[sl], 1u);
          else atomicOr(&pg.cnt[sl], 0x80000000u);
        }
        __threadfence();
        __syncthreads();
        for (int sl = tid; sl < kGH; sl += kBlock) {
          const uint64_t t = pg.tag[sl];
          if ((uint32_t)(t >> 32) != pg.gen) continue;
          const int id = (int)((uint32_t)t - 1u);
          const uint32_t hcv = pg.cnt[sl];
          const bool hb = (hcv >> 31) != 0u;
          float bsum = 0.0f;
          if (hb) {
            for (int e = 0; e < c.nbias; ++e)
              if (c.bias_ids[e] == id) bsum = bsum + c.bias_vals[e];
          }
          const bool allowed = !c.mask || ((((id >> 5) < Wm ? c.mask[id >> 5] : 0u) >> (id & 31)) & 1u);
          pg.fin[sl] = allowed ? fold_nan(penalised_key(load_elem_bits<DT>(c.xrow, id), c.mode, c.rep, c.freq,
                                                        c.pres, (int)(hcv & 0x7FFFFFFFu), hb, bsum))
                               : 0u;
        }
        __threadfence();
        __syncthreads();
      }
      ovf = 1u;  // the fast path uses the LDS table only
    }
  }

  // 3. candidate pool: elements whose composite is >= tc (fast path)
  int nT = 0;
  uint32_t tk = 0u, ti = 0u;
  bool slow = ovf != 0u;
  uint32_t plo = tmax, phi = hi;
  bool binned = false;  // sampling epilogue done on key bins
  int btoken = -1;
  float blogprob = 0.0f;
  if (!empty && want > 0) {
    uint32_t nfin = 0u;  // patched final values at the front of the pool
    uint32_t C = 0u;
    uint32_t Cv = 0u;  // valid pool elements (C less the invalidated raw copies)
    if (!slow) {
      nfin = nfin0;
      C = gather_pool<DT>(a, c, S, NG, pmode == 1, tc, pool, Cv, nfin, cur);
      if ((int)C > a.pcap || (int)Cv < want) slow = true;
      phi = max(hi, hfmax);  // every pool key lies in [tmax, phi]
    }
    if (!slow && want == 1) {  // greedy: the pool maximum
      uint64_t mc = 0ull;
      for (int i = tid; i < (int)C; i += kBlock)
        if (pool[i].x >= kKeyFloor) mc = max(mc, comp_of(pool[i].x, pool[i].y));
      mc = block_max(mc, S.r64);
      if (tid == 0) pool[0] = make_uint2(comp_key(mc), comp_idx(mc));
      lds_barrier();
      nT = 1;
    } else if (!slow) {
      // four pool entries per thread are loaded before any is used
      auto visit_pool = [&](auto&& f) {
        for (int i0 = tid; i0 < (int)C; i0 += 4 * kBlock) {
          uint2 e[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) e[u] = pool[i0 + u * kBlock < (int)C ? i0 + u * kBlock : 0];
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (i0 + u * kBlock < (int)C) f(e[u].x, e[u].y);
        }
      };
      if constexpr (sampling_op(OP) && DT == SS_BF16) {
        const bool ext = OP == OP_SAMPLE_X && (a.gum || c.full_row);  // these draw element-wise
        const uint32_t span = (phi >> 16) - (tmax >> 16);  // key values the pool spans
        if (!a.out_idx && !ext && span < (uint32_t)kBlock)
          binned = sample_binned<kBlock>(c, S, pool, (int)C, (int)nfin, (uint32_t)want, tmax >> 16, a.V, b, btoken,
                                         blogprob);
        else if (!a.out_idx && !ext && span < (uint32_t)kEBins)
          binned = sample_binned<kEBins>(c, S, pool, (int)C, (int)nfin, (uint32_t)want, tmax >> 16, a.V, b, btoken,
                                         blogprob);
      }
      if (binned) {
        nT = want;  // T is not materialised on this path
      } else {
        radix_select(visit_pool, (uint32_t)want, Cv, plo, phi, a.V, S, &tk, &ti);
        nT = (int)compact_pool(S, pool, (int)C, [&](uint2 e) { return selected(e.x, e.y, tk, ti); });
      }
    } else {
      flags |= SS_FLAG_FALLBACK;
      nT = slow_select<DT>(a, c, S, pool, NG, pmode, pg, want, &tk, &ti);
    }
  }
  lds_barrier();
  if (tid < kMaxU / 32) S.rmask[tid] = 0u;  // clean for the next merge of this workgroup
  const bool none = empty || nT == 0;
  if (!empty && nT == 0 && want > 0) flags |= SS_FLAG_EMPTY;  // every token masked or penalised to -inf

  // 4. row maximum (canonical first element) of the selection
  uint64_t mc = 0ull;
  uint32_t kmin = 0xFFFFFFFFu;
  if (!binned) {
    for (int i = tid; i < nT; i += kBlock) {
      mc = max(mc, comp_of(pool[i].x, pool[i].y));
      kmin = min(kmin, pool[i].x);
    }
    block_max_min(mc, kmin, S);
  }
  const uint64_t Mcomp = mc;
  const int argmax = none ? -1 : (int)comp_idx(Mcomp);
  if (empty) flags = SS_FLAG_EMPTY;
  if (none) flags |= SS_FLAG_EMPTY;

  if constexpr (OP == OP_TOPK) {
    const int n_sel = nT;
    if (n_sel > 0) {
      uint64_t* sel = reinterpret_cast<uint64_t*>(pool);
      const int N = next_pow2(n_sel);
      for (int i = tid; i < N; i += kBlock) {  // each slot converted by its own thread
        const uint64_t cm = i < n_sel ? comp_of(pool[i].x, pool[i].y) : 0ull;
        sel[i] = cm;
      }
      lds_barrier();
      lds_sort_desc(sel, N);
    }
    const uint64_t* sel = reinterpret_cast<const uint64_t*>(pool);
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
  } else if constexpr (OP == OP_LOGPROBS) {
    // the leading tokens in canonical order, then the full-row normaliser:
    // the units' sums (taken by the streaming kernel relative to each unit's
    // raw maximum) rescaled to the row maximum M, each patched id's raw term
    // replaced by its final value's
    const int n_sel = none ? 0 : nT;
    if (n_sel > 0) {
      uint64_t* sel = reinterpret_cast<uint64_t*>(pool);
      const int N = next_pow2(n_sel);
      for (int i = tid; i < N; i += kBlock) sel[i] = i < n_sel ? comp_of(pool[i].x, pool[i].y) : 0ull;
      lds_barrier();
      lds_sort_desc(sel, N);
    }
    const float tauf = lp_tau(a, c.mode, b);
    const double tau = (double)tauf;
    const double M = n_sel > 0 ? (double)float_of_key(comp_key(Mcomp)) : 0.0;
    double z = n_sel > 0 ? row_norm_part<DT>(a, c, S, row, pmode, pg, M, tauf) : 0.0;
    z = block_sum(z, S.rd);
    const double lz = n_sel > 0 ? log(z) : 0.0;
    const uint64_t* sel = reinterpret_cast<const uint64_t*>(pool);
    for (int r = tid; r < a.k_cap; r += kBlock) {
      const size_t o = (size_t)b * a.k_cap + r;
      if (r < n_sel) {
        a.out_idx[o] = (int32_t)comp_idx(sel[r]);
        a.out_val[o] = (float)(((double)float_of_key(comp_key(sel[r])) - M) / tau - lz);
      } else {
        a.out_idx[o] = -1;
        a.out_val[o] = -__builtin_inff();
      }
    }
    if (a.flags && tid == 0) a.flags[b] = (c.mode & SS_LOGPROBS) ? flags & (SS_FLAG_FALLBACK | SS_FLAG_EMPTY) : 0;
    return;
  } else {
    int token = -1;
    float logprob = 0.0f;
    int accept = 0;
    const int64_t pos = c.pos;
    const uint64_t seed = c.seed;
    bool has_draft = false;
    int dtok = -1;
    if constexpr (OP == OP_VERIFY) {
      if (c.ell < a.L) {
        dtok = c.dtok;
        has_draft = dtok >= 0 && dtok < a.V;
      }
    }
    if (OP == OP_PROCESS && a.patched && tid == 0) a.npatched[row] = 0u;
    if (OP == OP_PROCESS && pmode == 1) {
      // (id, final key) list for the materialising pass, in slot order
      uint32_t cnt = 0u;
      for (int sl = tid; sl < kH; sl += kBlock) cnt += S.hk[sl] >= 0 ? 1u : 0u;
      uint32_t tot;
      uint32_t off = block_excl_scan(cnt, S.r32, tot);
      for (int sl = tid; sl < kH; sl += kBlock)
        if (S.hk[sl] >= 0) a.patched[(size_t)row * kGH + off++] = make_uint2((uint32_t)S.hk[sl], S.hf[sl]);
      if (tid == 0) a.npatched[row] = tot;
    } else if (OP == OP_PROCESS && pmode == 2) {
      uint32_t cnt = 0u;
      for (int s = tid; s < kGH; s += kBlock) cnt += (uint32_t)(pg.tag[s] >> 32) == pg.gen ? 1u : 0u;
      uint32_t tot;
      uint32_t off = block_excl_scan(cnt, S.r32, tot);
      for (int s = tid; s < kGH; s += kBlock) {
        const uint64_t t = pg.tag[s];
        if ((uint32_t)(t >> 32) == pg.gen) a.patched[(size_t)row * kGH + off++] = make_uint2((uint32_t)t - 1u, pg.fin[s]);
      }
      if (tid == 0) a.npatched[row] = tot;
    } else if (OP == OP_PROCESS && pmode == 3) {
      if (tid == 0) a.npatched[row] = kLinear;
    }
    if (!none && c.greedy) {
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
      if constexpr (sampling_op(OP)) {
        if (a.out_idx) {
          for (int r = tid; r < a.k_out; r += kBlock) {
            a.out_idx[(size_t)b * a.k_out + r] = r == 0 ? argmax : -1;
            a.out_prob[(size_t)b * a.k_out + r] = r == 0 ? 1.0f : 0.0f;
          }
        }
      }
    } else if (binned) {
      token = btoken;
      logprob = blogprob;
    } else if (!none) {
      // ---- truncation and selection epilogue (Alg. 11 order) on T = pool[0, nT)
      const double M = (double)float_of_key(comp_key(Mcomp));
      const double tau = (double)c.tau;
      const double itau = 1.0 / tau;
      const bool minp = (c.mode & SS_MINP) && c.min_p > 0.0f;
      const bool topp = (c.mode & SS_TOPP) && c.top_p < 1.0f;
      const double lt = minp ? log((double)c.min_p) : 0.0;
      // weights of T in 2^-50 fixed point, stored behind T in the pool region
      uint64_t* Wl = reinterpret_cast<uint64_t*>(pool) + a.pcap / 2;
      const int MT = (nT + kBlock - 1) / kBlock;
      uint32_t inT = 0u, keepm = 0u;
      uint64_t zl = 0ull;
      for (int m = 0; m < MT; ++m) {
        const int i = tid + m * kBlock;
        if (i < nT) {
          const uint2 e = pool[i];
          const double y = (double)float_of_key(e.x);
          const uint64_t w = (uint64_t)__double2ll_rn(weight_fast(y, M, itau) * kFix);
          Wl[i] = w;
          zl += w;
          inT |= 1u << m;
          bool kp = true;
          if (minp && comp_of(e.x, e.y) != Mcomp) {
            const double l = (y == M) ? 0.0 : (y - M) / tau;
            kp = l >= lt;
          }
          if (kp) keepm |= 1u << m;
        }
      }
      const uint64_t Zk = block_sum(zl, S.r64);  // its barriers publish Wl
      // kept set S = T, min-p survivors, canonical prefix up to the top-p
      // boundary ep (the first element whose running mass reaches p * Z).
      // Full-row truncation (Appendix C.2) takes Z over the whole row; its
      // result stands when the kept set holds fewer than k_max tokens, else
      // the bounded one (Z over T) is taken with KCAP.
      double zthr = (double)Zk;
      bool full_try = OP == OP_SAMPLE_X && c.full_row;
      if (full_try)
        zthr = kFix * block_sum(row_norm_part<DT>(a, c, S, row, pmode, pg, M, lp_tau(a, c.mode, b)), S.rd);
      uint32_t inS = 0u;
      uint64_t zs = 0ull, lastc = ~0ull;
      uint32_t ns = 0u;
      uint32_t smin = 0xFFFFFFFFu;
      for (;;) {
        uint64_t ep = 0ull;
        if (topp) ep = cross_find(S, pool, Wl, nT, inT, (double)c.top_p * zthr, false, kmin, comp_key(Mcomp), a.V);
        inS = 0u;
        zs = 0ull;
        lastc = ~0ull;
        ns = 0u;
        smin = 0xFFFFFFFFu;
        for (int m = 0; m < MT; ++m) {
          const int i = tid + m * kBlock;
          if ((keepm >> m) & 1u) {
            const uint64_t cm = comp_of(pool[i].x, pool[i].y);
            if (ep == 0ull || cm >= ep) {
              inS |= 1u << m;
              zs += Wl[i];
              ++ns;
              lastc = min(lastc, cm);
              smin = min(smin, pool[i].x);
            }
          }
        }
        block_sum_min2(zs, lastc, ns, smin, S);
        if (!full_try) break;
        full_try = false;
        if (ns < (uint32_t)a.k_cap) {
          flags &= ~SS_FLAG_KCAP;
          break;
        }
        flags |= SS_FLAG_KCAP;
        zthr = (double)Zk;
      }
      const uint64_t Zs = zs;
      const uint32_t n_s = ns;
      const uint64_t last = lastc;
      const double Zsd = (double)Zs / kFix;
      const double u0 = uniform01(seed, (uint32_t)b, pos, 0);
      auto draw = [&](double total) -> uint64_t {
        const uint64_t e = cross_find(S, pool, Wl, nT, inS, u0 * total, true, smin, comp_key(Mcomp), a.V);
        return e == 0ull ? last : e;
      };
      if constexpr (OP == OP_PROCESS) {
        if (tid == 0) {
          RowSummary s;
          s.thr = last;
          s.Z = Zsd;
          s.M = (float)M;
          s.tau = (float)tau;
          s.argmax = argmax;
          s.kind = KIND_DIST;
          a.summ[row] = s;
        }
      } else {
        if (sampling_op(OP) || !has_draft) {
          uint64_t e;
          if (OP == OP_SAMPLE_X && a.gum) {
            // Gumbel-max over the kept set (Appendix C.3): the largest
            // (y - M)/tau - g[id] in double, the lower id on equal scores
            const float* grow = a.gum + (size_t)b * (size_t)a.ld_g;
            double bs = -__builtin_inf();
            uint64_t bk = 0ull;  // (~id << 32) | key of this thread's best
            for (int m = 0; m < MT; ++m) {
              if ((inS >> m) & 1u) {
                const int i = tid + m * kBlock;
                const double y = (double)float_of_key(pool[i].x);
                const double sc = (y == M ? 0.0 : (y - M) / tau) - (double)grow[pool[i].y];
                const uint64_t k2 = ((uint64_t)(~pool[i].y) << 32) | pool[i].x;
                if (sc > bs || (sc == bs && k2 > bk)) {
                  bs = sc;
                  bk = k2;
                }
              }
            }
            const double top = block_max(bs, S.rd);
            const uint64_t win = block_max<uint64_t>(bs == top ? bk : (uint64_t)0, S.r64);
            e = comp_of((uint32_t)win, ~(uint32_t)(win >> 32));
          } else {
            e = draw((double)Zs);
          }
          token = (int)comp_idx(e);
          const double w = weight_fast((double)float_of_key(comp_key(e)), M, itau);
          logprob = (float)log(w / Zsd);
          if constexpr (sampling_op(OP)) {
            if (a.out_idx) {
              // kept list in canonical order: compact S to the front, sort
              uint64_t* srt = reinterpret_cast<uint64_t*>(pool);
              for (int m = 0; m < MT; ++m) {
                const int i = tid + m * kBlock;
                if (i < nT && !((inS >> m) & 1u)) pool[i] = make_uint2(0u, 0u);
              }
              lds_barrier();
              const uint32_t tot = compact_pool(S, pool, nT, [](uint2 e2) { return e2.x != 0u; });
              const int N = next_pow2((int)tot);
              for (int i = tid; i < N; i += kBlock) {
                const uint64_t cm = i < (int)tot ? comp_of(pool[i].x, pool[i].y) : 0ull;
                srt[i] = cm;
              }
              lds_barrier();
              lds_sort_desc(srt, N);
              for (int rr = tid; rr < a.k_out; rr += kBlock) {
                if (rr < (int)n_s) {
                  const uint64_t cc = srt[rr];
                  a.out_idx[(size_t)b * a.k_out + rr] = (int32_t)comp_idx(cc);
                  a.out_prob[(size_t)b * a.k_out + rr] =
                      (float)(weight_fast((double)float_of_key(comp_key(cc)), M, itau) / Zsd);
                } else {
                  a.out_idx[(size_t)b * a.k_out + rr] = -1;
                  a.out_prob[(size_t)b * a.k_out + rr] = 0.0f;
                }
              }
              if ((int)n_s > a.k_out) flags |= SS_FLAG_OUT_TRUNC;
            }
          }
        } else {
          // verification of draft token dtok against this row's distribution
          const float* qrow = a.draft_probs ? a.draft_probs + ((size_t)b * a.L + c.ell) * (size_t)a.ld_q : nullptr;
          double pd_local = 0.0;
          for (int m = 0; m < MT; ++m) {
            const int i = tid + m * kBlock;
            if (((inS >> m) & 1u) && (int)pool[i].y == dtok)
              pd_local = weight_fast((double)float_of_key(pool[i].x), M, itau) / Zsd;
          }
          const double Pd = block_max(pd_local, S.rd);
          // sparse q: the entries naming an id summed, an unlisted id at 0
          const bool sparse = a.kq > 0;
          const size_t qo = ((size_t)b * a.L + c.ell) * (size_t)a.kq;
          uint64_t* ql = qlist_view(S);
          int NQ = 0;
          double qd;
          if (sparse) {
            // the list into LDS as (id << 32 | q bits), ids outside [0, V)
            // as 0xFFFFFFFF, padded to a power of two when it will be sorted
            NQ = a.kq <= kQScan ? a.kq : next_pow2(a.kq);
            double qs = 0.0;
            for (int i = tid; i < NQ; i += kBlock) {
              uint64_t e = ~0ull;
              if (i < a.kq) {
                const int id = a.dq_idx[qo + i];
                const float v = a.dq_val[qo + i];
                if (id == dtok) qs += (double)v;
                if (id >= 0 && id < a.V) e = ((uint64_t)(uint32_t)id << 32) | __float_as_uint(v);
              }
              ql[i] = e;
            }
            qd = block_sum(qs, S.rd);  // its barriers publish the list
          } else {
            qd = (double)qrow[dtok];
          }
          const double u1 = uniform01(seed, (uint32_t)b, pos, 1);
          accept = (Pd > 0.0 && u1 * qd <= Pd) ? 1 : 0;
          // a long list is sorted (ids descending, padding first) for binary
          // search; a short one is scanned in list order, every lane reading
          // the same entry
          const bool qsorted = sparse && !accept && a.kq > kQScan;
          if (qsorted) lds_sort_desc(ql, NQ);
          auto q_of = [&](uint32_t id) -> double {
            if (!sparse) return (double)qrow[id];
            double s = 0.0;
            if (!qsorted) {
#pragma unroll 8
              for (int j = 0; j < NQ; ++j) {
                const uint64_t e = ql[j];
                if ((uint32_t)(e >> 32) == id) s += (double)__uint_as_float((uint32_t)e);
              }
              return s;
            }
            int lo = 0, hi = NQ;  // first entry whose id is at most `id`
            while (lo < hi) {
              const int mid = (lo + hi) >> 1;
              if ((uint32_t)(ql[mid] >> 32) > id) lo = mid + 1;
              else hi = mid;
            }
            for (; lo < NQ && (uint32_t)(ql[lo] >> 32) == id; ++lo) s += (double)__uint_as_float((uint32_t)ql[lo]);
            return s;
          };
          if (!accept) {
            // residual max(0, P - q) over the kept set, canonical order, in
            // place of the kept weights (restored when the residual is empty)
            uint64_t rl = 0ull;
            for (int m = 0; m < MT; ++m) {
              if ((inS >> m) & 1u) {
                const int i = tid + m * kBlock;
                const double P = weight_fast((double)float_of_key(pool[i].x), M, itau) / Zsd;
                const double v = P - q_of(pool[i].y);
                const uint64_t r = v > 0.0 ? (uint64_t)__double2ll_rn(v * kFix) : 0ull;
                Wl[i] = r;
                rl += r;
              }
            }
            const uint64_t Rt = block_sum(rl, S.r64);  // its barriers publish the residuals
            uint64_t e;
            if (Rt > 0ull) {
              e = draw((double)Rt);
            } else {
              for (int m = 0; m < MT; ++m) {
                if ((inS >> m) & 1u) {
                  const int i = tid + m * kBlock;
                  Wl[i] = (uint64_t)__double2ll_rn(weight_fast((double)float_of_key(pool[i].x), M, itau) * kFix);
                }
              }
              lds_barrier();
              e = draw((double)Zs);
            }
            token = (int)comp_idx(e);
          }
        }
      }
    }

    if constexpr (OP == OP_PROCESS) {
      if (none && tid == 0) {
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
    } else if constexpr (sampling_op(OP)) {
      if (tid == 0) {
        a.out_token[b] = token;
        if (a.out_logprob) a.out_logprob[b] = logprob;
        if (a.flags) a.flags[b] = flags;
      }
      if (none && a.out_idx) {
        for (int r = tid; r < a.k_out; r += kBlock) {
          a.out_idx[(size_t)b * a.k_out + r] = -1;
          a.out_prob[(size_t)b * a.k_out + r] = 0.0f;
        }
      }
      return;
    } else {
      // publish this row's decision; the assembly kernel combines a request's rows
      if (tid == 0) {
        RowResult rr;
        rr.accept = accept;
        rr.emit = token;
        rr.flags = flags;
        rr.pad = 0;
        a.res[row] = rr;
      }
    }
  }
}

// ===========================================================================
// Patch tables (workgroups of the streaming launch)
// ===========================================================================
struct PSmem {
  int32_t hk[kH];   // listed id (or -1)
  uint32_t hc[kH];  // occurrence count | has-bias bit 31 | duplicate-bias bit 30
  uint32_t hf[kH];  // bias value, then the final key
  uint32_t flagsw;  // nonzero: more distinct ids than kH slots
  uint32_t pad[3];
};

// Builds a row's patch table: the history, draft and bias ids are counted and
// summed in an LDS hash table (bias entries of one id summed in list order),
// each listed id's raw logit is gathered and its final key computed by the
// Appendix C.1 prologue (Alg. 8 order; grammar-masked ids get the invalid
// key).  The table goes to the workspace slot for slot, with the row's
// status: 0 no lists, 1 table written, 2 more distinct ids than the table
// holds (the merge then builds a table in global memory itself).  It needs
// the logits and the lists only, so it runs beside the row stream.
template <int DT>
__device__ __forceinline__ void patch_row(const KArgs& a, int row, PSmem& P) {
  const int tid = threadIdx.x;
  const Ctx c = make_ctx<DT>(a, row);
  const int ne = c.nhist + c.nextra + c.nbias;
  if (ne == 0) {
    if (tid == 0) a.pstat[row] = 0;
    return;
  }
  int hid0[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const int h = tid + m * kSBlock;
    hid0[m] = h < c.nhist ? c.hist[h] : -1;
  }
  const int bid0 = tid < c.nbias ? c.bias_ids[tid] : -1;
  const float bval0 = tid < c.nbias ? c.bias_vals[tid] : 0.0f;
  for (int sl = tid; sl < kH / 4; sl += kSBlock) {
    reinterpret_cast<int4*>(P.hk)[sl] = make_int4(-1, -1, -1, -1);
    reinterpret_cast<uint4*>(P.hc)[sl] = make_uint4(0u, 0u, 0u, 0u);
  }
  if (tid == 0) P.flagsw = 0u;
  lds_barrier();
  // a second bias entry for one id sets the "duplicate" bit; the finals then
  // sum that id's entries in list order
  auto ins = [&](int id, uint32_t addc, bool bias, float bval) {
    if (id < 0 || id >= a.V) return;
    uint32_t sl = hslot(id);
    for (int p = 0; p < kProbe; ++p) {
      const int old = atomicCAS(&P.hk[sl], -1, id);
      if (old == -1 || old == id) {
        if (addc) atomicAdd(&P.hc[sl], addc);
        if (bias) {
          const uint32_t prev = atomicOr(&P.hc[sl], 0x80000000u);
          if (prev & 0x80000000u) atomicOr(&P.hc[sl], 0x40000000u);
          else P.hf[sl] = __float_as_uint(bval);
        }
        return;
      }
      sl = (sl + 1) & (kH - 1);
    }
    P.flagsw = 1u;
  };
#pragma unroll
  for (int m = 0; m < 4; ++m) ins(hid0[m], 1u, false, 0.0f);
  for (int h = tid + 4 * kSBlock; h < c.nhist; h += kSBlock) ins(c.hist[h], 1u, false, 0.0f);  // long histories
  for (int h = tid; h < c.nextra; h += kSBlock) ins(c.extra[h], 1u, false, 0.0f);
  ins(bid0, 0u, true, bval0);
  for (int e = tid + kSBlock; e < c.nbias; e += kSBlock) ins(c.bias_ids[e], 0u, true, c.bias_vals[e]);
  lds_barrier();
  if (P.flagsw != 0u) {
    if (tid == 0) a.pstat[row] = 2;
    return;
  }
  // final keys: every slot's raw logit (and grammar word) is loaded before
  // any is used
  constexpr int kSl = kH / kSBlock;
  const int Wm = (a.V + 31) >> 5;
  int id[kSl];
  uint32_t bits[kSl], mw[kSl];
#pragma unroll
  for (int m = 0; m < kSl; ++m) {
    id[m] = P.hk[tid + m * kSBlock];
    const int ld = id[m] >= 0 ? id[m] : 0;  // element 0 stands in for an empty slot
    bits[m] = load_elem_bits<DT>(c.xrow, ld);
    mw[m] = c.mask ? ((ld >> 5) < Wm ? c.mask[ld >> 5] : 0u) : 0xFFFFFFFFu;
  }
  uint32_t* dst = a.ptab + (size_t)row * 2 * kH;
#pragma unroll
  for (int m = 0; m < kSl; ++m) {
    const int sl = tid + m * kSBlock;
    uint32_t k = 0u;
    if (id[m] >= 0) {
      const uint32_t hcv = P.hc[sl];
      const bool hb = (hcv >> 31) != 0u;
      float bsum = 0.0f;
      if (hb) {
        if (hcv & 0x40000000u) {  // duplicate bias ids: list order
          for (int e = 0; e < c.nbias; ++e)
            if (c.bias_ids[e] == id[m]) bsum = bsum + c.bias_vals[e];
        } else {
          bsum = 0.0f + __uint_as_float(P.hf[sl]);
        }
      }
      if ((mw[m] >> (id[m] & 31)) & 1u)
        k = fold_nan(penalised_key(bits[m], c.mode, c.rep, c.freq, c.pres, (int)(hcv & 0x3FFFFFFFu), hb, bsum));
    }
    dst[sl] = (uint32_t)id[m];
    dst[kH + sl] = k;
  }
  if (tid == 0) a.pstat[row] = 1;
}

// ===========================================================================
// Kernels
// ===========================================================================
// Streaming kernel: one unit per wavefront, no LDS, no barrier.  Workgroups
// are remapped so that consecutive units (one row) share an XCD and its L2.
// For the operations that apply penalties and bias, the first workgroups of
// the grid build the rows' patch tables (dynamic LDS) beside the stream.
template <int DT, bool LP>
__global__ __launch_bounds__(kSBlock) void ss_stream_kernel(KArgs a) {
  int bid = blockIdx.x;
  if (bid < a.patch_wgs) {  // patch-table workgroups (a multiple of 8) come first
    extern __shared__ __align__(16) unsigned char psmem[];
    // on the XCD that streams the row (below), so the gathers of its listed
    // ids and its units' loads share that XCD's L2
    int row = bid;
    if ((a.rows & 7) == 0 && ((a.rows * a.U) & 31) == 0) row = (bid & 7) * (a.rows >> 3) + (bid >> 3);
    if (row < a.rows) patch_row<DT>(a, row, *reinterpret_cast<PSmem*>(psmem));
    return;
  }
  bid -= a.patch_wgs;
  const int nb = gridDim.x - a.patch_wgs;
  if (bid < (nb & ~7)) bid = (bid & 7) * (nb >> 3) + (bid >> 3);
  const int gu = __builtin_amdgcn_readfirstlane(bid * kSWaves + wave());
  if (gu < a.rows * a.U) scan_unit<DT, LP>(a, gu);
}

// Merge kernel: one workgroup per row (the launch boundary orders the
// streaming kernel's records and candidates before it).
template <int DT, int OP>
__global__ __launch_bounds__(kBlock) void ss_merge_kernel(KArgs a) {
  extern __shared__ __align__(16) unsigned char smem_raw[];
  MSmem& S = *reinterpret_cast<MSmem*>(smem_raw);
  uint2* pool = reinterpret_cast<uint2*>(smem_raw + kSmemFixed);
  if (threadIdx.x < kMaxU / 32) S.rmask[threadIdx.x] = 0u;
  __syncthreads();
  // The streaming kernel placed row r's units on XCD floor(8 r / rows) when
  // its grid splits evenly over the 8 XCDs; the same remap here runs the
  // row's merge on that XCD as well.
  int row = blockIdx.x;
  const int nunits = a.rows * a.U;
  if ((a.rows & 7) == 0 && (nunits & 31) == 0) row = (row & 7) * (a.rows >> 3) + (row >> 3);
  merge_row<DT, OP>(a, row, S, pool);
}

// Verification assembly: per request, the accepted drafts, then the first


// ---------------------------------------------------------------------------
// Materialising pass of ss_process_logits: processed logits and final
// probabilities for every element, from the per-row summary; patched ids take
// their final values from the merge's list.
// ---------------------------------------------------------------------------
template <int DT>
__global__ __launch_bounds__(kBlock) void ss_materialize_kernel(KArgs a) {
  constexpr int TILE = 4096;
  const int tid = threadIdx.x;
  const int T = (a.V + TILE - 1) / TILE;
  const int row = blockIdx.x / T;
  const int tile = blockIdx.x - row * T;
  const int lo = tile * TILE;
  const int hi = min(a.V, lo + TILE);
  const int b = row;
  const uint32_t mode = (a.mode ? a.mode[b] : 0u) & a.feat;
  const uint32_t* mask = (mode & SS_GRAMMAR) ? a.bitmask + (size_t)row * (size_t)a.mask_ld : nullptr;
  const unsigned char* xrow = reinterpret_cast<const unsigned char*>(a.x) + (size_t)row * (size_t)a.ld * DTT<DT>::ES;
  const RowSummary s = a.summ[row];
  const double sitau = 1.0 / (double)s.tau;
  const size_t ob = (size_t)row * (size_t)a.V;
  const int Wm = (a.V + 31) >> 5;
  auto emit = [&](uint32_t k, uint32_t i) {
    if (a.out_logits) a.out_logits[ob + i] = k >= kKeyFloor ? float_of_key(k) : -__builtin_inff();
    if (a.out_probs) {
      float p = 0.0f;
      if (s.kind == KIND_GREEDY) {
        p = (int)i == s.argmax ? 1.0f : 0.0f;
      } else if (s.kind == KIND_DIST && k >= kKeyFloor && comp_of(k, i) >= s.thr) {
        p = (float)(weight_fast((double)float_of_key(k), (double)s.M, sitau) / s.Z);
      }
      a.out_probs[ob + i] = p;
    }
  };
  // final keys of the patched ids of this tile, staged in LDS (kNone elsewhere)
  constexpr uint32_t kNone = 0xFFFFFFFFu;
  __shared__ uint32_t pv[TILE];
  for (int l = tid; l < TILE; l += kBlock) pv[l] = kNone;
  __syncthreads();
  const uint32_t np = a.npatched ? a.npatched[row] : 0u;
  const uint2* pl = a.patched + (size_t)row * kGH;
  for (uint32_t j = tid; np != kLinear && j < np; j += kBlock) {
    const uint2 e = pl[j];
    if ((int)e.x >= lo && (int)e.x < hi) pv[e.x - lo] = e.y;
  }
  __syncthreads();
  for (int i = lo + tid; i < hi; i += kBlock) {
    uint32_t k = fold_nan(key_raw(load_elem_bits<DT>(xrow, i)));
    if (mask && !((((i >> 5) < Wm ? mask[i >> 5] : 0u) >> (i & 31)) & 1u)) k = 0u;
    const uint32_t pk = pv[i - lo];
    if (pk != kNone) k = pk;
    if (np == kLinear) {  // very long lists: look every id up
      const Ctx c = make_ctx<DT>(a, row);
      int cn;
      bool hb;
      float bs;
      if (lin_info(c, i, &cn, &hb, &bs) && k != 0u) k = lin_final<DT>(a, c, i);
    }
    emit(k, (uint32_t)i);
  }
}

}  // namespace ss
