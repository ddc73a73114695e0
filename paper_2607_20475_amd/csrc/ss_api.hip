// ss_api.hip -- host side of libss.so: workspace layout, argument validation,
// launch sequence and the C ABI declared in ss.h.
#include "ss_impl.hpp"
#include "ss_launch.hpp"

namespace ss {

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
struct Layout {
  int U, cap, pcap, rows, smem;
  size_t off_rec, off_cand, off_res, off_patch, off_npatch, off_gtag, off_gcnt, off_gfin,
      off_pstat, off_ptab, off_usum, total;
};

static size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

static bool make_layout(int op, int B, int V, int L, int k_max, int dtype, Layout* lay) {
  if (B <= 0 || V <= 0 || V > SS_MAX_V || k_max < 1 || k_max > SS_MAX_K) return false;
  if (op == OP_VERIFY && (L < 1 || L > SS_MAX_L)) return false;
  if (op < OP_TOPK || op > OP_LOGPROBS) return false;
  const int rows = op == OP_VERIFY ? B * (L + 1) : B;
  const int U = (V + kUE - 1) / kUE;
  const int cap = unit_cap(k_max, U, dtype);
  // pool entries: candidates; after selection T in the front half and, for
  // the sampling ops, its fixed-point weights in the back half
  int pcap = 2 * k_max + 128;
  if (pcap < 1024) pcap = 1024;
  if (pcap < next_pow2(k_max)) pcap = next_pow2(k_max);
  pcap = (pcap + 255) & ~255;
  size_t o = 0;
  lay->off_rec = o;
  o = align256(o + (size_t)rows * U * 16);
  lay->off_cand = o;
  o = align256(o + (size_t)rows * U * cap * 16);
  lay->off_res = o;
  const size_t res_bytes = op == OP_VERIFY ? sizeof(RowResult) : (op == OP_PROCESS ? sizeof(RowSummary) : 0);
  o = align256(o + (size_t)rows * res_bytes);
  lay->off_patch = o;
  if (op == OP_PROCESS) o = align256(o + (size_t)rows * kGH * 8);
  lay->off_npatch = o;
  if (op == OP_PROCESS) o = align256(o + (size_t)rows * 4);
  const size_t ghr = op == OP_TOPK ? 0 : (size_t)rows;  // top-k applies no penalties
  lay->off_gtag = o;
  o = align256(o + ghr * kGH * 8);
  lay->off_gcnt = o;
  o = align256(o + ghr * kGH * 4);
  lay->off_gfin = o;
  o = align256(o + ghr * kGH * 4);
  // patch tables built by the streaming launch: status word and 2 kH words per row
  lay->off_pstat = o;
  o = align256(o + ghr * 4);
  lay->off_ptab = o;
  o = align256(o + ghr * 2 * kH * 4);
  // log-probabilities and full-row sampling: every unit's share of its row's normaliser
  lay->off_usum = o;
  if (op == OP_LOGPROBS || op == OP_SAMPLE) o = align256(o + (size_t)rows * U * 8);
  lay->total = o;
  lay->U = U;
  lay->cap = cap;
  lay->pcap = pcap;
  lay->rows = rows;
  lay->smem = kSmemFixed + 8 * (pcap + kBlock);  // pool plus one dump slot per thread
  return true;
}

static uint32_t feature_mask(const ss_params* p) {
  uint32_t f = SS_GREEDY | SS_GRAMMAR | SS_REP | SS_FREQ | SS_PRES | SS_BIAS | SS_TEMP | SS_TOPK | SS_TOPP | SS_MINP |
               SS_LOGPROBS;
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

// The merge instantiation of a call: sampling with full-row truncation or the
// Gumbel-max draw has its own, so plain sampling carries neither extension.
static int merge_op(const KArgs& k) { return (k.op == OP_SAMPLE && (k.full || k.gum)) ? (int)OP_SAMPLE_X : k.op; }

static void launch_merge_any(const KArgs& k, int dtype, dim3 grid, dim3 block, int smem, hipStream_t st) {
  if (dtype == SS_BF16) {
    switch (merge_op(k)) {
      case OP_TOPK: launch_merge<SS_BF16, OP_TOPK>(k, grid, block, smem, st); break;
      case OP_SAMPLE: launch_merge<SS_BF16, OP_SAMPLE>(k, grid, block, smem, st); break;
      case OP_VERIFY: launch_merge<SS_BF16, OP_VERIFY>(k, grid, block, smem, st); break;
      case OP_LOGPROBS: launch_merge<SS_BF16, OP_LOGPROBS>(k, grid, block, smem, st); break;
      case OP_SAMPLE_X: launch_merge<SS_BF16, OP_SAMPLE_X>(k, grid, block, smem, st); break;
      default: launch_merge<SS_BF16, OP_PROCESS>(k, grid, block, smem, st); break;
    }
  } else {
    switch (merge_op(k)) {
      case OP_TOPK: launch_merge<SS_F32, OP_TOPK>(k, grid, block, smem, st); break;
      case OP_SAMPLE: launch_merge<SS_F32, OP_SAMPLE>(k, grid, block, smem, st); break;
      case OP_VERIFY: launch_merge<SS_F32, OP_VERIFY>(k, grid, block, smem, st); break;
      case OP_LOGPROBS: launch_merge<SS_F32, OP_LOGPROBS>(k, grid, block, smem, st); break;
      case OP_SAMPLE_X: launch_merge<SS_F32, OP_SAMPLE_X>(k, grid, block, smem, st); break;
      default: launch_merge<SS_F32, OP_PROCESS>(k, grid, block, smem, st); break;
    }
  }
}

static hipError_t merge_smem_any(int dtype, int op, int bytes) {
  if (dtype == SS_BF16) {
    switch (op) {
      case OP_TOPK: return merge_smem_limit<SS_BF16, OP_TOPK>(bytes);
      case OP_SAMPLE: return merge_smem_limit<SS_BF16, OP_SAMPLE>(bytes);
      case OP_VERIFY: return merge_smem_limit<SS_BF16, OP_VERIFY>(bytes);
      case OP_LOGPROBS: return merge_smem_limit<SS_BF16, OP_LOGPROBS>(bytes);
      case OP_SAMPLE_X: return merge_smem_limit<SS_BF16, OP_SAMPLE_X>(bytes);
      default: return merge_smem_limit<SS_BF16, OP_PROCESS>(bytes);
    }
  }
  switch (op) {
    case OP_TOPK: return merge_smem_limit<SS_F32, OP_TOPK>(bytes);
    case OP_SAMPLE: return merge_smem_limit<SS_F32, OP_SAMPLE>(bytes);
    case OP_VERIFY: return merge_smem_limit<SS_F32, OP_VERIFY>(bytes);
    case OP_LOGPROBS: return merge_smem_limit<SS_F32, OP_LOGPROBS>(bytes);
    case OP_SAMPLE_X: return merge_smem_limit<SS_F32, OP_SAMPLE_X>(bytes);
    default: return merge_smem_limit<SS_F32, OP_PROCESS>(bytes);
  }
}

static bool smem_configured[2][6];

static ss_status launch(KArgs& k, int dtype, const Layout& lay, void* ws, hipStream_t st, bool materialize) {
  unsigned char* w = reinterpret_cast<unsigned char*>(ws);
  k.U = lay.U;
  k.cap = lay.cap;
  k.pcap = lay.pcap;
  k.rec = reinterpret_cast<uint4*>(w + lay.off_rec);
  k.cand = reinterpret_cast<uint4*>(w + lay.off_cand);
  k.res = reinterpret_cast<RowResult*>(w + lay.off_res);
  k.summ = reinterpret_cast<RowSummary*>(w + lay.off_res);
  k.patched = k.op == OP_PROCESS ? reinterpret_cast<uint2*>(w + lay.off_patch) : nullptr;
  k.npatched = k.op == OP_PROCESS ? reinterpret_cast<uint32_t*>(w + lay.off_npatch) : nullptr;
  k.gtag = reinterpret_cast<uint64_t*>(w + lay.off_gtag);
  k.gcnt = reinterpret_cast<uint32_t*>(w + lay.off_gcnt);
  k.gfin = reinterpret_cast<uint32_t*>(w + lay.off_gfin);
  k.pstat = reinterpret_cast<int32_t*>(w + lay.off_pstat);
  k.ptab = reinterpret_cast<uint32_t*>(w + lay.off_ptab);
  k.usum = (k.op == OP_LOGPROBS || k.full) ? reinterpret_cast<double*>(w + lay.off_usum) : nullptr;
  // patch-table workgroups (a multiple of 8, so the stream's XCD remap holds)
  k.patch_wgs = k.op == OP_TOPK ? 0 : (lay.rows + 7) & ~7;
  const int di = dtype == SS_BF16 ? 1 : 0;
  const int mop = merge_op(k);
  if (!smem_configured[di][mop]) {
    // the largest dynamic LDS any call can ask for
    const int maxb = kSmemFixed + 8 * (((2 * SS_MAX_K + 128 + 255) & ~255) + kBlock);
    if (merge_smem_any(dtype, mop, maxb) != hipSuccess) return SS_ERR_HIP;
    smem_configured[di][mop] = true;
  }
  const int nunits = lay.rows * lay.U;
  const dim3 grid((unsigned)(k.patch_wgs + (nunits + kSWaves - 1) / kSWaves)), sblock(kSBlock),
      rgrid((unsigned)lay.rows), block(kBlock);
  const int psmem = k.patch_wgs ? (int)sizeof(PSmem) : 0;
  const bool lp = k.op == OP_LOGPROBS || k.full;  // units add their normaliser shares
  if (dtype == SS_BF16)
    lp ? launch_stream<SS_BF16, true>(k, grid, sblock, psmem, st) : launch_stream<SS_BF16, false>(k, grid, sblock, psmem, st);
  else
    lp ? launch_stream<SS_F32, true>(k, grid, sblock, psmem, st) : launch_stream<SS_F32, false>(k, grid, sblock, psmem, st);
  launch_merge_any(k, dtype, rgrid, block, lay.smem, st);
  if (k.op == OP_VERIFY) launch_assemble(k, dim3((unsigned)((k.B + kBlock - 1) / kBlock)), block, st);
  if (materialize) {
    const int T = (k.V + 4095) / 4096;
    const dim3 mgrid((unsigned)(lay.rows * T));
    if (dtype == SS_BF16)
      launch_materialize<SS_BF16>(k, mgrid, block, st);
    else
      launch_materialize<SS_F32>(k, mgrid, block, st);
  }
  return hipGetLastError() == hipSuccess ? SS_OK : SS_ERR_HIP;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

static bool params_ok(const ss_params* p, int B, int V) {
  if (!p || p->B != B || p->V != V || !p->mode) return false;
  if (p->bitmask && p->bitmask_ld < (int64_t)((V + 31) / 32)) return false;
  return true;
}

}  // namespace ss

using namespace ss;

extern "C" {

size_t ss_workspace_bytes(int op, int B, int V, int L, int k_max, int dtype) {
  if (dtype != SS_F32 && dtype != SS_BF16) return 0;
  Layout lay;
  if (!make_layout(op, B, V, L, k_max, dtype, &lay)) return 0;
  return lay.total;
}

ss_status ss_workspace_init(void* ws, size_t ws_bytes, void* stream) {
  if (!ws || (ws_bytes & 3u) || !aligned16(ws)) return SS_ERR_INVALID_ARG;
  const size_t n = ws_bytes / 4;
  if (n == 0) return SS_OK;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  launch_zero(reinterpret_cast<uint32_t*>(ws), n, dim3((unsigned)blocks), dim3(256), (hipStream_t)stream);
  return hipGetLastError() == hipSuccess ? SS_OK : SS_ERR_HIP;
}

ss_status ss_topk(const void* x, int dtype, int B, int V, int64_t ld, const int32_t* k, int k_max, float* out_val,
                  int32_t* out_idx, int32_t* flags, void* ws, size_t ws_bytes, void* stream) {
  if (!x || !out_val || !out_idx || !ws || (dtype != SS_F32 && dtype != SS_BF16) || ld < V) return SS_ERR_INVALID_ARG;
  Layout lay;
  if (!make_layout(OP_TOPK, B, V, 0, k_max, dtype, &lay)) return SS_ERR_INVALID_ARG;
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

ss_status ss_logprobs(const void* logits, int dtype, int64_t ld, const ss_params* p, int n_lp, int32_t* out_idx,
                      float* out_lp, int32_t* flags, void* ws, size_t ws_bytes, void* stream) {
  if (!logits || !p || !out_idx || !out_lp || !ws || (dtype != SS_F32 && dtype != SS_BF16)) return SS_ERR_INVALID_ARG;
  const int B = p->B, V = p->V;
  if (ld < V || !params_ok(p, B, V)) return SS_ERR_INVALID_ARG;
  Layout lay;
  if (!make_layout(OP_LOGPROBS, B, V, 0, n_lp, dtype, &lay)) return SS_ERR_INVALID_ARG;
  if (ws_bytes < lay.total || !aligned16(ws)) return SS_ERR_WORKSPACE;
  KArgs a = {};
  a.x = logits;
  a.ld = ld;
  a.op = OP_LOGPROBS;
  a.B = B;
  a.rows = B;
  a.V = V;
  a.L = 0;
  a.k_cap = n_lp;
  a.vec_ok = aligned16(logits) && ((ld * esize(dtype)) % 16 == 0);
  fill_params(a, p);
  a.out_idx = out_idx;
  a.out_val = out_lp;
  a.flags = flags;
  return launch(a, dtype, lay, ws, (hipStream_t)stream, false);
}

static ss_status sample_any(const void* logits, int dtype, int64_t ld, const ss_params* p, int k_max, int full,
                            const float* noise, int64_t ld_noise, int32_t* out_token, float* out_logprob,
                            int32_t* out_idx, float* out_prob, int k_out, int32_t* flags, void* ws, size_t ws_bytes,
                            void* stream) {
  if (!logits || !p || !out_token || !ws || (dtype != SS_F32 && dtype != SS_BF16)) return SS_ERR_INVALID_ARG;
  if (k_out < 0 || (k_out > 0 && (!out_idx || !out_prob))) return SS_ERR_INVALID_ARG;
  const int B = p->B, V = p->V;
  if (ld < V || !params_ok(p, B, V)) return SS_ERR_INVALID_ARG;
  if (noise && ld_noise < V) return SS_ERR_INVALID_ARG;
  Layout lay;
  if (!make_layout(OP_SAMPLE, B, V, 0, k_max, dtype, &lay)) return SS_ERR_INVALID_ARG;
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
  a.gum = noise;
  a.ld_g = noise ? ld_noise : 0;
  a.full = full;
  a.out_token = out_token;
  a.out_logprob = out_logprob;
  a.out_idx = k_out > 0 ? out_idx : nullptr;
  a.out_prob = k_out > 0 ? out_prob : nullptr;
  a.flags = flags;
  return launch(a, dtype, lay, ws, (hipStream_t)stream, false);
}

ss_status ss_sample(const void* logits, int dtype, int64_t ld, const ss_params* p, int k_max, int32_t* out_token,
                    float* out_logprob, int32_t* out_idx, float* out_prob, int k_out, int32_t* flags, void* ws,
                    size_t ws_bytes, void* stream) {
  return sample_any(logits, dtype, ld, p, k_max, 0, nullptr, 0, out_token, out_logprob, out_idx, out_prob, k_out,
                    flags, ws, ws_bytes, stream);
}

ss_status ss_sample_full(const void* logits, int dtype, int64_t ld, const ss_params* p, int k_max,
                         int32_t* out_token, float* out_logprob, int32_t* out_idx, float* out_prob, int k_out,
                         int32_t* flags, void* ws, size_t ws_bytes, void* stream) {
  return sample_any(logits, dtype, ld, p, k_max, 1, nullptr, 0, out_token, out_logprob, out_idx, out_prob, k_out,
                    flags, ws, ws_bytes, stream);
}

ss_status ss_sample_gumbel(const void* logits, int dtype, int64_t ld, const ss_params* p, int k_max,
                           const float* noise, int64_t ld_noise, int32_t* out_token, float* out_logprob,
                           int32_t* out_idx, float* out_prob, int k_out, int32_t* flags, void* ws, size_t ws_bytes,
                           void* stream) {
  if (!noise) return SS_ERR_INVALID_ARG;
  return sample_any(logits, dtype, ld, p, k_max, 0, noise, ld_noise, out_token, out_logprob, out_idx, out_prob,
                    k_out, flags, ws, ws_bytes, stream);
}

static ss_status verify_any(const void* target_logits, int dtype, int64_t ld_row, int Lt, const int32_t* row_map,
                            const float* draft_probs, int64_t ld_q, const int32_t* q_idx, const float* q_val, int kq,
                            const int32_t* draft_tokens, int L, const ss_params* p, int k_max, int32_t* out_tokens,
                            int32_t* out_num_accepted, int32_t* flags, void* ws, size_t ws_bytes, void* stream) {
  if (!target_logits || !p || !draft_tokens || !out_tokens || !out_num_accepted || !ws) return SS_ERR_INVALID_ARG;
  if (dtype != SS_F32 && dtype != SS_BF16) return SS_ERR_INVALID_ARG;
  const int B = p->B, V = p->V;
  if (ld_row < V || !params_ok(p, B, V)) return SS_ERR_INVALID_ARG;
  if (kq == 0 && (!draft_probs || ld_q < V)) return SS_ERR_INVALID_ARG;
  if (kq != 0 && (!q_idx || !q_val || kq < 1 || kq > SS_MAX_K)) return SS_ERR_INVALID_ARG;
  if (row_map && Lt < 1) return SS_ERR_INVALID_ARG;
  if (!p->seed || !p->position) return SS_ERR_INVALID_ARG;
  Layout lay;
  if (!make_layout(OP_VERIFY, B, V, L, k_max, dtype, &lay)) return SS_ERR_INVALID_ARG;
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
  a.draft_probs = kq == 0 ? draft_probs : nullptr;
  a.ld_q = kq == 0 ? ld_q : 0;
  a.dq_idx = q_idx;
  a.dq_val = q_val;
  a.kq = kq;
  a.rmap = row_map;
  a.Lt = row_map ? Lt : L + 1;
  a.draft_tokens = draft_tokens;
  a.out_tokens = out_tokens;
  a.out_nacc = out_num_accepted;
  a.flags = flags;
  return launch(a, dtype, lay, ws, (hipStream_t)stream, false);
}

ss_status ss_verify(const void* target_logits, int dtype, int64_t ld_row, const float* draft_probs, int64_t ld_q,
                    const int32_t* draft_tokens, int L, const ss_params* p, int k_max, int32_t* out_tokens,
                    int32_t* out_num_accepted, int32_t* flags, void* ws, size_t ws_bytes, void* stream) {
  return verify_any(target_logits, dtype, ld_row, L + 1, nullptr, draft_probs, ld_q, nullptr, nullptr, 0,
                    draft_tokens, L, p, k_max, out_tokens, out_num_accepted, flags, ws, ws_bytes, stream);
}

ss_status ss_verify_sparse(const void* target_logits, int dtype, int64_t ld_row, const int32_t* draft_idx,
                           const float* draft_q, int kq, const int32_t* draft_tokens, int L, const ss_params* p,
                           int k_max, int32_t* out_tokens, int32_t* out_num_accepted, int32_t* flags, void* ws,
                           size_t ws_bytes, void* stream) {
  if (kq < 1 || kq > SS_MAX_K || !draft_idx || !draft_q) return SS_ERR_INVALID_ARG;
  return verify_any(target_logits, dtype, ld_row, L + 1, nullptr, nullptr, 0, draft_idx, draft_q, kq, draft_tokens,
                    L, p, k_max, out_tokens, out_num_accepted, flags, ws, ws_bytes, stream);
}

ss_status ss_verify_tree(const void* target_logits, int dtype, int64_t ld_row, int Lt, const int32_t* row_map,
                         const int32_t* draft_idx, const float* draft_q, int kq, const int32_t* draft_tokens, int L,
                         const ss_params* p, int k_max, int32_t* out_tokens, int32_t* out_num_accepted,
                         int32_t* flags, void* ws, size_t ws_bytes, void* stream) {
  if (!row_map || Lt < 1 || kq < 1 || kq > SS_MAX_K || !draft_idx || !draft_q) return SS_ERR_INVALID_ARG;
  return verify_any(target_logits, dtype, ld_row, Lt, row_map, nullptr, 0, draft_idx, draft_q, kq, draft_tokens, L,
                    p, k_max, out_tokens, out_num_accepted, flags, ws, ws_bytes, stream);
}

ss_status ss_process_logits(const void* logits, int dtype, int64_t ld, const ss_params* p, int k_max,
                            float* out_logits, float* out_probs, int32_t* flags, void* ws, size_t ws_bytes,
                            void* stream) {
  if (!logits || !p || !ws || (dtype != SS_F32 && dtype != SS_BF16)) return SS_ERR_INVALID_ARG;
  const int B = p->B, V = p->V;
  if (ld < V || !params_ok(p, B, V)) return SS_ERR_INVALID_ARG;
  Layout lay;
  if (!make_layout(OP_PROCESS, B, V, 0, k_max, dtype, &lay)) return SS_ERR_INVALID_ARG;
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