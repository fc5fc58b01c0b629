// C ABI of the BSA library: argument validation, buffer carving and the launch order of
// the forward pass on the caller's stream. Declarations and contracts: include/bsa.h.
#include "../../include/bsa.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <map>
#include <mutex>
#include <string>

#include "kernels.hpp"

namespace {

thread_local std::string g_last_error;

bsa_status_t fail(bsa_status_t s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

bool pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

bsa_status_t hip_status(hipError_t e, const char* where) {
  if (e == hipSuccess) return BSA_OK;
  return fail(BSA_ERR_HIP, std::string(where) + ": " + hipGetErrorString(e));
}

#define BSA_TRY(expr, where)                         \
  do {                                               \
    bsa_status_t _s = hip_status((expr), (where));   \
    if (_s != BSA_OK) return _s;                     \
  } while (0)

// Validate p and fill the internal sizes.
bsa_status_t check_params(const bsa_params_t* p, bsa::Dims* D) {
  if (!p) return fail(BSA_ERR_INVALID_ARGUMENT, "params is NULL");
  if (p->batch < 1 || p->heads < 1) return fail(BSA_ERR_INVALID_ARGUMENT, "batch and heads must be >= 1");
  if (!pow2(p->n) || p->n < 64 || p->n > (1 << 24))
    return fail(BSA_ERR_INVALID_ARGUMENT, "n must be a power of two in [64, 2^24]");
  if (p->head_dim != 32 && p->head_dim != 64) return fail(BSA_ERR_UNSUPPORTED, "head_dim must be 32 or 64");
  if (!pow2(p->ball_size) || p->ball_size < 64 || p->ball_size > p->n)
    return fail(BSA_ERR_INVALID_ARGUMENT, "ball_size must be a power of two in [64, n]");
  if (!pow2(p->cmp_block) || p->n / p->cmp_block < 16)
    return fail(BSA_ERR_INVALID_ARGUMENT, "cmp_block must be a power of two with n/cmp_block >= 16");
  if (p->cmp_stride != p->cmp_block)
    return fail(BSA_ERR_UNSUPPORTED, "cmp_stride must equal cmp_block (non-overlapping blocks, Eq. 5)");
  if (p->slc_block % 16 != 0 || p->slc_block % p->cmp_block != 0 || p->ball_size % p->slc_block != 0)
    return fail(BSA_ERR_INVALID_ARGUMENT, "slc_block must be a multiple of 16 and of cmp_block and divide ball_size");
  const int r = p->slc_block / p->cmp_block;
  if (r != 1 && r != 2 && r != 4) return fail(BSA_ERR_UNSUPPORTED, "slc_block / cmp_block must be 1, 2 or 4");
  if (!pow2(p->group_size) || p->ball_size % p->group_size != 0)
    return fail(BSA_ERR_INVALID_ARGUMENT, "group_size must be a power of two dividing ball_size");
  if (p->group_size != 1 && p->group_size < 8)
    return fail(BSA_ERR_UNSUPPORTED, "group_size must be 1 (per-token selection) or >= 8");
  if (p->group_size == 1 && p->dtype != BSA_BF16)
    return fail(BSA_ERR_UNSUPPORTED, "per-token selection (group_size 1) needs bf16 storage");
  if (p->topk < 1 || p->topk > 16) return fail(BSA_ERR_UNSUPPORTED, "topk must be in [1, 16]");
  const int G = p->group_size >= 16 ? 1 : 16 / p->group_size;
  if (p->group_size >= 8 && G * p->topk * (p->slc_block / 16) > 256)
    return fail(BSA_ERR_UNSUPPORTED, "too many selected tokens per 16-query block (limit 4096)");
  if ((int64_t)p->batch * p->heads * p->n * p->topk >= (int64_t)1 << 31)
    return fail(BSA_ERR_UNSUPPORTED, "batch * heads * n * topk must stay below 2^31");
  if (p->mask_own_ball != 0 && p->mask_own_ball != 1) return fail(BSA_ERR_INVALID_ARGUMENT, "mask_own_ball must be 0/1");
  if (p->store_lse != 0 && p->store_lse != 1) return fail(BSA_ERR_INVALID_ARGUMENT, "store_lse must be 0/1");
  if (p->deterministic != 0 && p->deterministic != 1) return fail(BSA_ERR_INVALID_ARGUMENT, "deterministic must be 0/1");
  if (p->kv_pool != BSA_POOL_MLP && p->kv_pool != BSA_POOL_MEAN) return fail(BSA_ERR_INVALID_ARGUMENT, "bad kv_pool");
  if (p->kv_pool == BSA_POOL_MLP && (p->cmp_block * p->head_dim) % 64 != 0)
    return fail(BSA_ERR_UNSUPPORTED, "MLP pooling needs cmp_block * head_dim to be a multiple of 64");
  if (p->dtype != BSA_F32 && p->dtype != BSA_BF16) return fail(BSA_ERR_INVALID_ARGUMENT, "bad dtype");
  if (p->dtype == BSA_F32 && p->head_dim != 32)
    return fail(BSA_ERR_UNSUPPORTED, "float32 layers support head_dim 32 (bf16 layers: 32 and 64)");
  if (!(p->softmax_scale >= 0.0f) || std::isinf(p->softmax_scale))
    return fail(BSA_ERR_INVALID_ARGUMENT, "softmax_scale must be finite and >= 0");
  if (p->q_coarsen != BSA_QC_MEAN && p->q_coarsen != BSA_QC_MLP) return fail(BSA_ERR_INVALID_ARGUMENT, "bad q_coarsen");
  if (p->group_compression != 0 && p->group_compression != 1)
    return fail(BSA_ERR_INVALID_ARGUMENT, "group_compression must be 0/1");
  if ((p->q_coarsen == BSA_QC_MLP || p->group_compression) && p->group_size != p->cmp_block)
    return fail(BSA_ERR_INVALID_ARGUMENT,
                "block query coarsening (Eq. 13) and group compression (Eq. 15) need group_size == cmp_block");
  if (p->q_coarsen == BSA_QC_MLP && (p->cmp_block * p->head_dim) % 64 != 0)
    return fail(BSA_ERR_UNSUPPORTED, "MLP query coarsening needs cmp_block * head_dim to be a multiple of 64");
  if (p->group_compression && p->n / p->cmp_block < 64)
    return fail(BSA_ERR_UNSUPPORTED, "group compression needs n / cmp_block >= 64");
  D->B = p->batch;
  D->H = p->heads;
  D->N = p->n;
  D->d = p->head_dim;
  D->m = p->ball_size;
  D->l = p->cmp_block;
  D->ls = p->slc_block;
  D->k = p->topk;
  D->g = p->group_size;
  D->mask_own = p->mask_own_ball;
  D->pool = p->kv_pool;
  D->bf16 = p->dtype == BSA_BF16;
  D->qc_mlp = p->q_coarsen == BSA_QC_MLP;
  D->gcmp = p->group_compression;
  D->store_lse = p->store_lse;
  D->scale = p->softmax_scale > 0.f ? p->softmax_scale : 1.0f / std::sqrt((float)p->head_dim);
  return BSA_OK;
}

size_t elem_bytes(const bsa::Dims& D) { return D.bf16 ? 2 : 4; }

struct SavedLayout {
  size_t sel, lse, ob, ocf, kc, vc, hk, hv, cv, qc, hq, oc, total;
};

SavedLayout saved_layout(const bsa::Dims& D) {
  SavedLayout L{};
  const size_t rows = (size_t)D.rows();
  const size_t crows = (size_t)D.cmp_rows();
  size_t off = 0;
  auto put = [&](size_t bytes) { size_t o = off; off += align256(bytes); return o; };
  L.sel = put(sizeof(int32_t) * (size_t)D.B * D.H * (D.N / D.g) * D.k);
  L.lse = put(D.store_lse ? sizeof(float) * 3 * rows : 0);
  L.ob = put(elem_bytes(D) * 2 * rows * D.d);
  L.ocf = put(sizeof(float) * rows * D.d);
  L.kc = put(sizeof(float) * crows * D.d);
  L.vc = put(sizeof(float) * crows * D.d);
  L.hk = put(sizeof(float) * crows * D.d);
  L.hv = put(sizeof(float) * crows * D.d);
  L.cv = put((size_t)D.B * (D.N / D.l));
  L.qc = put(sizeof(float) * (size_t)D.B * D.H * (D.N / D.g) * D.d);
  L.hq = put(D.qc_mlp ? sizeof(float) * crows * D.d : 0);
  L.oc = put(D.gcmp ? sizeof(float) * crows * D.d : 0);
  L.total = off;
  return L;
}

struct FwdWs {
  size_t w1t_k, w1t_v, w1t_q, kc_lp, vc_lp, qc_lp, lsec, kplanes, lse;
  size_t pk, pv, pkt, pvt, hist, seg_s, seg_e, part, ml;   // per-token selection (g = 1)
  size_t total;
};

// Per-token selection buffers: sorted (query, slot) pairs, block ranges, partials.
bsa::Slc1Ws slc1_ws(const bsa::Dims& D, char* w, size_t pk, size_t pv, size_t pkt, size_t pvt, size_t hist,
                    size_t seg_s, size_t seg_e, size_t part, size_t ml) {
  bsa::Slc1Ws W{};
  W.keys = (uint32_t*)(w + pk);
  W.vals = (uint32_t*)(w + pv);
  W.keys_tmp = (uint32_t*)(w + pkt);
  W.vals_tmp = (uint32_t*)(w + pvt);
  W.hist = (uint32_t*)(w + hist);
  W.seg_start = (int*)(w + seg_s);
  W.seg_end = (int*)(w + seg_e);
  W.part = (float*)(w + part);
  W.ml = ml == (size_t)-1 ? nullptr : (float*)(w + ml);
  (void)D;
  return W;
}

FwdWs fwd_ws_layout(const bsa::Dims& D) {
  FwdWs W{};
  size_t off = 0;
  auto put = [&](size_t bytes) { size_t o = off; off += align256(bytes); return o; };
  const size_t w1 = elem_bytes(D) * (size_t)D.l * D.d * D.d;
  W.w1t_k = put(w1);
  W.w1t_v = put(w1);
  W.kc_lp = put(elem_bytes(D) * (size_t)D.cmp_rows() * D.d);
  W.vc_lp = put(elem_bytes(D) * (size_t)D.cmp_rows() * D.d);
  W.w1t_q = put(D.qc_mlp ? w1 : 0);
  W.qc_lp = put(D.block_coarse() ? elem_bytes(D) * (size_t)D.cmp_rows() * D.d : 0);
  W.lsec = put(D.gcmp ? sizeof(float) * (size_t)D.cmp_rows() : 0);
  W.kplanes = put(3 * sizeof(uint16_t) * (size_t)D.cmp_rows() * D.d);
  W.lse = put(D.store_lse ? 0 : sizeof(float) * 3 * (size_t)D.rows());   // not kept: forward scratch
  const size_t np = D.g == 1 ? bsa::slc1_pairs(D) : 0;
  const size_t nseg = D.g == 1 ? (size_t)D.B * D.H * (D.N / D.ls) : 0;
  W.pk = put(4 * np);
  W.pv = put(4 * np);
  W.pkt = put(4 * np);
  W.pvt = put(4 * np);
  W.hist = put(D.g == 1 ? 4 * bsa::radix_sort_hist_words((long long)np) : 0);
  W.seg_s = put(4 * nseg);
  W.seg_e = put(4 * nseg);
  W.part = put(sizeof(float) * np * D.d);
  W.ml = put(2 * sizeof(float) * np);
  W.total = off;
  return W;
}

struct BwdWs {
  size_t qc_lp, doc, t4c, dqc, dqpart, lse, lsec, ml;
  size_t R, terms, dplp, kc_lp, vc_lp, dkc_part, dvc_part, dkc, dvc, pk, pv, pkt, pvt, hist, seg_s, seg_e, dpre, pw1, psm, w1lp,
      total;
  int cmp_chunks, mlp_chunks, mlp_chunks_small;
  long long pairs, nseg;
};

BwdWs bwd_ws_layout(const bsa::Dims& D) {
  BwdWs W{};
  size_t off = 0;
  auto put = [&](size_t bytes) { size_t o = off; off += align256(bytes); return o; };
  const size_t rows = (size_t)D.rows();
  const size_t crows = (size_t)D.cmp_rows();
  W.cmp_chunks = D.N / 8 >= 64 ? 8 : 1;
  W.mlp_chunks = bsa::mlp_bwd_chunks(D);
  W.mlp_chunks_small = bsa::mlp_bwd_chunks_small(D);
  W.pairs = (long long)D.B * D.H * (D.N / D.g) * D.k;
  W.nseg = (long long)D.B * D.H * (D.N / D.ls);
  W.R = put(sizeof(float) * 3 * rows);
  W.terms = put(sizeof(float) * 4 * 3 * rows);
  W.kc_lp = put(elem_bytes(D) * crows * D.d);
  W.vc_lp = put(elem_bytes(D) * crows * D.d);
  W.dkc_part = put(sizeof(float) * W.cmp_chunks * crows * D.d);
  W.dvc_part = put(sizeof(float) * W.cmp_chunks * crows * D.d);
  W.dkc = put(sizeof(float) * crows * D.d);
  W.dvc = put(sizeof(float) * crows * D.d);
  W.pk = put(4 * (size_t)W.pairs);
  W.pv = put(4 * (size_t)W.pairs);
  W.pkt = put(4 * (size_t)W.pairs);
  W.pvt = put(4 * (size_t)W.pairs);
  W.hist = put(4 * bsa::radix_sort_hist_words(W.pairs));
  W.seg_s = put(4 * (size_t)W.nseg);
  W.seg_e = put(4 * (size_t)W.nseg);
  W.dpre = put(sizeof(float) * crows * D.d);
  W.pw1 = put(sizeof(float) * (size_t)W.mlp_chunks * D.l * D.d * D.d);
  W.psm = put(sizeof(float) * (size_t)W.mlp_chunks_small * ((size_t)D.d * D.d + 2 * D.d));
  W.w1lp = put(elem_bytes(D) * (size_t)D.l * D.d * D.d);
  W.dplp = put(elem_bytes(D) * crows * D.d);
  W.qc_lp = put(D.gcmp ? elem_bytes(D) * crows * D.d : 0);
  W.doc = put(D.gcmp ? elem_bytes(D) * crows * D.d : 0);
  W.t4c = put(D.gcmp ? 4 * sizeof(float) * crows : 0);
  W.dqc = put(D.gcmp ? sizeof(float) * crows * D.d : 0);
  W.dqpart = put(D.g == 1 ? sizeof(float) * bsa::slc1_pairs(D) * D.d : 0);
  // store_lse = 0: recomputed log-sum-exp rows (and what their recomputation needs)
  W.lse = put(D.store_lse ? 0 : sizeof(float) * 3 * rows);
  W.lsec = put(!D.store_lse && D.gcmp ? sizeof(float) * crows : 0);
  W.ml = put(!D.store_lse && D.g == 1 ? 2 * sizeof(float) * bsa::slc1_pairs(D) : 0);
  W.total = off;
  return W;
}

}  // namespace

extern "C" {

const char* bsa_status_string(bsa_status_t s) {
  switch (s) {
    case BSA_OK: return "ok";
    case BSA_ERR_INVALID_ARGUMENT: return "invalid argument";
    case BSA_ERR_UNSUPPORTED: return "unsupported";
    case BSA_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case BSA_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char* bsa_last_error(void) { return g_last_error.c_str(); }

bsa_status_t bsa_timing_enable(int32_t on) {
  g_last_error.clear();
  bsa::timing_set(on != 0);
  return BSA_OK;
}

bsa_status_t bsa_timing_select(const char* phases) {
  g_last_error.clear();
  bsa::timing_select(phases);
  return BSA_OK;
}

bsa_status_t bsa_timing_query(const char* phase, double* total_ms, int32_t* count) {
  g_last_error.clear();
  if (!phase || !total_ms || !count) return fail(BSA_ERR_INVALID_ARGUMENT, "phase, total_ms and count must be non-NULL");
  int n = 0;
  BSA_TRY(bsa::timing_query(phase, total_ms, &n), "bsa_timing_query");
  *count = n;
  return BSA_OK;
}

size_t bsa_ball_tree_workspace_bytes(int64_t n_real, int64_t n_pad, int32_t dim, int32_t batch) {
  if (n_real < 1 || n_real > n_pad || !pow2(n_pad) || n_pad > (1 << 24) || dim < 1 || dim > 3 || batch < 1) return 0;
  if ((int64_t)batch * n_pad > (int64_t(1) << 30)) return 0;
  return bsa::tree_workspace_bytes(n_real, n_pad, batch);
}

bsa_status_t bsa_build_ball_tree(const float* points, int64_t n_real, int32_t dim, int64_t n_pad, int32_t batch,
                                 int32_t* perm, void* ws, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  if (!points || !perm) return fail(BSA_ERR_INVALID_ARGUMENT, "points and perm must be non-NULL");
  if (dim < 1 || dim > 3) return fail(BSA_ERR_UNSUPPORTED, "dim must be 1, 2 or 3");
  if (batch < 1) return fail(BSA_ERR_INVALID_ARGUMENT, "batch must be >= 1");
  if (!pow2(n_pad) || n_pad > (1 << 24)) return fail(BSA_ERR_INVALID_ARGUMENT, "n_pad must be a power of two <= 2^24");
  if (n_real < 1 || n_real > n_pad) return fail(BSA_ERR_INVALID_ARGUMENT, "need 1 <= n_real <= n_pad");
  const size_t need = bsa_ball_tree_workspace_bytes(n_real, n_pad, dim, batch);
  if (need == 0) return fail(BSA_ERR_INVALID_ARGUMENT, "batch * n_pad too large");
  if (!ws || ws_bytes < need)
    return fail(BSA_ERR_WORKSPACE_TOO_SMALL, "tree workspace needs " + std::to_string(need) + " bytes");
  hipError_t e;
  BSA_PHASE("tree", (hipStream_t)stream,
            e = bsa::launch_build_tree(points, n_real, dim, n_pad, batch, perm, ws, (hipStream_t)stream));
  BSA_TRY(e, "bsa_build_ball_tree");
  return BSA_OK;
}

bsa_status_t bsa_build_ball_tree_noalloc(const float* points, int64_t n_real, int32_t dim, int64_t n_pad,
                                         int32_t batch, int32_t* perm, void* stream) {
  g_last_error.clear();
  if (!points || !perm) return fail(BSA_ERR_INVALID_ARGUMENT, "points and perm must be non-NULL");
  if (dim < 1 || dim > 3) return fail(BSA_ERR_UNSUPPORTED, "dim must be 1, 2 or 3");
  if (batch < 1) return fail(BSA_ERR_INVALID_ARGUMENT, "batch must be >= 1");
  if (!pow2(n_pad) || n_pad > (1 << 24)) return fail(BSA_ERR_INVALID_ARGUMENT, "n_pad must be a power of two <= 2^24");
  if (n_real < 1 || n_real > n_pad) return fail(BSA_ERR_INVALID_ARGUMENT, "need 1 <= n_real <= n_pad");
  if ((int64_t)batch * n_pad > bsa::tree_scratch_slots())
    return fail(BSA_ERR_UNSUPPORTED, "batch * n_pad = " + std::to_string((int64_t)batch * n_pad) +
                                         " exceeds the allocation-free tree build's limit of " +
                                         std::to_string(bsa::tree_scratch_slots()) +
                                         " slots; use bsa_build_ball_tree with a workspace");
  if (bsa_ball_tree_workspace_bytes(n_real, n_pad, dim, batch) > bsa::tree_scratch_bytes())
    return fail(BSA_ERR_UNSUPPORTED, "tree workspace exceeds the static scratch");
  void* scratch = nullptr;
  BSA_TRY(bsa::tree_scratch(&scratch), "bsa_build_ball_tree_noalloc (scratch address)");
  hipError_t e;
  BSA_PHASE("tree", (hipStream_t)stream,
            e = bsa::launch_build_tree(points, n_real, dim, n_pad, batch, perm, scratch, (hipStream_t)stream));
  BSA_TRY(e, "bsa_build_ball_tree_noalloc");
  return BSA_OK;
}

static bsa_status_t permute_common(const void* src, const int32_t* perm, int64_t n_real, int64_t n_pad, int32_t batch,
                                   int32_t heads, int32_t head_dim, int32_t dtype, void* dst) {
  if (!src || !perm || !dst) return fail(BSA_ERR_INVALID_ARGUMENT, "src, perm and dst must be non-NULL");
  if (batch < 1 || heads < 1 || head_dim < 1) return fail(BSA_ERR_INVALID_ARGUMENT, "batch, heads, head_dim >= 1");
  if (n_real < 1 || n_real > n_pad || n_pad > (1 << 24)) return fail(BSA_ERR_INVALID_ARGUMENT, "need 1 <= n_real <= n_pad <= 2^24");
  if (dtype != BSA_F32 && dtype != BSA_BF16) return fail(BSA_ERR_INVALID_ARGUMENT, "bad dtype");
  return BSA_OK;
}

bsa_status_t bsa_permute(const void* src, const int32_t* perm, int64_t n_real, int64_t n_pad, int32_t batch,
                         int32_t heads, int32_t head_dim, int32_t dtype, void* dst, uint8_t* valid_out, void* stream) {
  g_last_error.clear();
  bsa_status_t s = permute_common(src, perm, n_real, n_pad, batch, heads, head_dim, dtype, dst);
  if (s != BSA_OK) return s;
  hipError_t e;
  BSA_PHASE("permute", (hipStream_t)stream,
            e = bsa::launch_permute(src, perm, n_real, n_pad, batch, heads, head_dim, dtype, dst, valid_out, false,
                                    (hipStream_t)stream));
  BSA_TRY(e, "bsa_permute");
  return BSA_OK;
}

bsa_status_t bsa_unpermute(const void* src, const int32_t* perm, int64_t n_real, int64_t n_pad, int32_t batch,
                           int32_t heads, int32_t head_dim, int32_t dtype, void* dst, void* stream) {
  g_last_error.clear();
  bsa_status_t s = permute_common(src, perm, n_real, n_pad, batch, heads, head_dim, dtype, dst);
  if (s != BSA_OK) return s;
  BSA_TRY(bsa::launch_permute(src, perm, n_real, n_pad, batch, heads, head_dim, dtype, dst, nullptr, true,
                              (hipStream_t)stream),
          "bsa_unpermute");
  return BSA_OK;
}

bsa_status_t bsa_sizes(const bsa_params_t* p, size_t* ws_fwd_bytes, size_t* ws_bwd_bytes, size_t* saved_bytes) {
  g_last_error.clear();
  bsa::Dims D;
  bsa_status_t s = check_params(p, &D);
  if (s != BSA_OK) return s;
  if (ws_fwd_bytes) *ws_fwd_bytes = fwd_ws_layout(D).total;
  if (ws_bwd_bytes) *ws_bwd_bytes = bwd_ws_layout(D).total;
  if (saved_bytes) *saved_bytes = saved_layout(D).total;
  return BSA_OK;
}

bsa_status_t bsa_saved_view(const bsa_params_t* p, void* base, bsa_saved_t* out) {
  g_last_error.clear();
  bsa::Dims D;
  bsa_status_t s = check_params(p, &D);
  if (s != BSA_OK) return s;
  if (!base || !out) return fail(BSA_ERR_INVALID_ARGUMENT, "base and out must be non-NULL");
  SavedLayout L = saved_layout(D);
  char* c = (char*)base;
  out->sel_idx = (int32_t*)(c + L.sel);
  out->lse = D.store_lse ? (float*)(c + L.lse) : nullptr;
  out->o_branch = (void*)(c + L.ob);
  out->o_cmp = (float*)(c + L.ocf);
  out->kcmp = (float*)(c + L.kc);
  out->vcmp = (float*)(c + L.vc);
  out->hid_k = (float*)(c + L.hk);
  out->hid_v = (float*)(c + L.hv);
  out->cvalid = (uint8_t*)(c + L.cv);
  out->qcmp = (float*)(c + L.qc);
  out->hid_q = D.qc_mlp ? (float*)(c + L.hq) : nullptr;
  out->ocmp = D.gcmp ? (float*)(c + L.oc) : nullptr;
  return BSA_OK;
}

// One auxiliary stream (default priority) and a fork/join event pair per device, created on
// first use: independent branches run on it concurrently with the caller's stream. The
// mutex is held while a call enqueues its work, so the shared events are never recorded
// by two calls at once.
struct Aux {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};
std::mutex g_aux_mu;
std::map<int, Aux> g_aux;
int g_streams = 2;   // 1: every branch on the caller's stream; 0: also no shared launches (bsa_set_streams)

static bsa_status_t get_aux(Aux* out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return fail(BSA_ERR_HIP, "hipGetDevice failed");
  auto it = g_aux.find(dev);
  if (it == g_aux.end()) {
    Aux a;
    if (hipStreamCreateWithFlags(&a.s, hipStreamNonBlocking) != hipSuccess ||
        hipEventCreateWithFlags(&a.fork, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&a.join, hipEventDisableTiming) != hipSuccess)
      return fail(BSA_ERR_HIP, "creating the auxiliary stream and events failed");
    it = g_aux.emplace(dev, a).first;
  }
  *out = it->second;
  return BSA_OK;
}

static bsa_status_t join_aux(const Aux& a, hipStream_t st) {
  if (a.s == st) return BSA_OK;
  if (hipEventRecord(a.join, a.s) != hipSuccess || hipStreamWaitEvent(st, a.join, 0) != hipSuccess)
    return fail(BSA_ERR_HIP, "joining the auxiliary stream failed");
  return BSA_OK;
}

// Joins the auxiliary stream back into the caller's on every exit after a fork, so that a
// call that fails part-way still leaves no kernel of its own running past the caller's
// stream (it may still read the caller's buffers). join() does it early on the normal path.
struct AuxJoin {
  const Aux& a;
  hipStream_t st;
  bool armed = true;
  AuxJoin(const Aux& a_, hipStream_t st_) : a(a_), st(st_) {}
  bsa_status_t join() {
    armed = false;
    return join_aux(a, st);
  }
  ~AuxJoin() {
    if (armed && a.s != st) {
      (void)hipEventRecord(a.join, a.s);
      (void)hipStreamWaitEvent(st, a.join, 0);
    }
  }
};

bsa_status_t bsa_set_streams(int32_t n) {
  g_last_error.clear();
  if (n < 0 || n > 2) return fail(BSA_ERR_INVALID_ARGUMENT, "streams must be 0, 1 or 2");
  std::lock_guard<std::mutex> lock(g_aux_mu);
  g_streams = n;
  return BSA_OK;
}

static bool saved_ok(const bsa_saved_t* sv, const bsa::Dims& D) {
  return sv && sv->sel_idx && (sv->lse || !D.store_lse) && sv->o_branch && sv->o_cmp && sv->kcmp && sv->vcmp && sv->hid_k && sv->hid_v &&
         sv->cvalid && sv->qcmp && (!D.qc_mlp || sv->hid_q) && (!D.gcmp || sv->ocmp);
}

static bool mlp_ok(const bsa_mlp_t* m) { return m && m->w1 && m->b1 && m->w2 && m->b2; }

bsa_status_t bsa_forward(const bsa_params_t* p, const void* q, const void* k, const void* v, const uint8_t* valid,
                         const float* gate, const bsa_mlp_t* phi_k, const bsa_mlp_t* phi_v, const bsa_mlp_t* phi_q,
                         void* o, const bsa_saved_t* saved, void* ws, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  bsa::Dims D;
  bsa_status_t s = check_params(p, &D);
  if (s != BSA_OK) return s;
  if (!q || !k || !v || !gate || !o) return fail(BSA_ERR_INVALID_ARGUMENT, "q, k, v, gate and o must be non-NULL");
  if (!saved_ok(saved, D)) return fail(BSA_ERR_INVALID_ARGUMENT, "every saved buffer must be non-NULL");
  if (D.pool == 0 && (!mlp_ok(phi_k) || !mlp_ok(phi_v)))
    return fail(BSA_ERR_INVALID_ARGUMENT, "MLP pooling needs phi_k and phi_v with all four tensors");
  if (D.qc_mlp && !mlp_ok(phi_q))
    return fail(BSA_ERR_INVALID_ARGUMENT, "MLP query coarsening needs phi_q with all four tensors");
  const FwdWs W = fwd_ws_layout(D);
  if (!ws || ws_bytes < W.total)
    return fail(BSA_ERR_WORKSPACE_TOO_SMALL, "forward workspace needs " + std::to_string(W.total) + " bytes");
  hipStream_t st = (hipStream_t)stream;
  std::lock_guard<std::mutex> lock(g_aux_mu);
  Aux aux;
  s = get_aux(&aux);
  if (s != BSA_OK) return s;
  // the shared ball + compressed launch fills every CU (registers and LDS) until its tail,
  // so selection on a second stream would only wait beside it: one stream then
  const bool shared = valid == nullptr && g_streams != 0 && bsa::ball_cmp_fwd_fits(D);
  if (g_streams < 2 || shared) aux.s = st;
  char* w = (char*)ws;
  const size_t rows = (size_t)D.rows();
  char* ob = (char*)saved->o_branch;
  // store_lse = 0 with no saved buffer: the log-sum-exp rows go to forward scratch
  float* lse = saved->lse ? saved->lse : (float*)(w + W.lse);
  const size_t ob_stride = rows * D.d * elem_bytes(D);
  bsa::Mlp mk{}, mv{}, mq{};
  if (D.pool == 0) {
    mk = {phi_k->w1, phi_k->b1, phi_k->w2, phi_k->b2};
    mv = {phi_v->w1, phi_v->b1, phi_v->w2, phi_v->b2};
  }
  if (D.qc_mlp) mq = {phi_q->w1, phi_q->b1, phi_q->w2, phi_q->b2};
  bsa::Dims Dq = D;   // coarse queries of Eq. 13: phi_q (MLP) or the block mean
  Dq.pool = D.qc_mlp ? 0 : 1;
  void* kc_lp = w + W.kc_lp;
  void* vc_lp = w + W.vc_lp;
  void* qc_lp = w + W.qc_lp;
  hipError_t e = hipSuccess;
#define BSA_STEP(name, call, what)        \
  BSA_PHASE(name, st, e = (call));         \
  BSA_TRY(e, what)
  // keys and values in one launch
  const bsa::CompressJob kv_jobs[2] = {
      {k, mk, saved->kcmp, saved->hid_k, kc_lp, w + W.w1t_k, bsa::cmp_key_scale(D)},
      {v, mv, saved->vcmp, saved->hid_v, vc_lp, w + W.w1t_v, 1.0f}};
  BSA_STEP("fwd.compress", (bsa::launch_block_valid(D, valid, saved->cvalid, st) != hipSuccess
                                ? hipGetLastError()
                                : bsa::launch_compress_fwd(D, kv_jobs, 2, valid, st)),
           "compression");
  if (D.block_coarse()) {
    const bsa::CompressJob q_job = {q, mq, saved->qcmp, saved->hid_q, qc_lp, w + W.w1t_q, 1.0f};
    BSA_STEP("fwd.compress", bsa::launch_compress_fwd(Dq, &q_job, 1, valid, st), "query coarsening");
  }
  // ball and compressed attention on the auxiliary stream (the caller's one with the shared
  // launch), selection on the caller's
  if (aux.s != st &&
      (hipEventRecord(aux.fork, st) != hipSuccess || hipStreamWaitEvent(aux.s, aux.fork, 0) != hipSuccess))
    return fail(BSA_ERR_HIP, "forking the auxiliary stream failed");
  AuxJoin joiner(aux, st);
  {
    hipStream_t st_main = st;
    hipStream_t st = aux.s;
    if (shared) {
      BSA_STEP("fwd.ball_cmp",
               bsa::launch_ball_cmp_fwd(D, q, k, v, kc_lp, vc_lp, ob, lse, saved->o_cmp, lse + rows, st),
               "ball and compressed attention");
    } else {
      BSA_STEP("fwd.ball", bsa::launch_ball_fwd(D, q, k, v, valid, ob, lse, st), "ball attention");
      if (D.gcmp) {
        float* oc = saved->ocmp;
        float* lsec = (float*)(w + W.lsec);
        const uint8_t* cv = valid ? saved->cvalid : nullptr;
        BSA_STEP("fwd.cmp",
                 (bsa::launch_cmp_coarse_fwd(D, qc_lp, kc_lp, vc_lp, cv, oc, lsec, st) != hipSuccess
                      ? hipGetLastError()
                      : bsa::launch_expand_coarse(D, oc, lsec, valid, saved->o_cmp, lse + rows, st)),
                 "group compression");
      } else {
        BSA_STEP("fwd.cmp",
                 bsa::launch_cmp_fwd(D, q, kc_lp, vc_lp, valid, valid ? saved->cvalid : nullptr, saved->o_cmp,
                                     lse + rows, st),
                 "compressed attention");
      }
    }
    (void)st_main;
  }
  BSA_STEP("fwd.select", bsa::launch_select_topk(D, q, valid, saved->kcmp, saved->cvalid, saved->sel_idx,
                                                  saved->qcmp, D.block_coarse(), (uint16_t*)(w + W.kplanes), st),
           "select");
  if (D.g == 1) {
    const bsa::Slc1Ws S1 = slc1_ws(D, w, W.pk, W.pv, W.pkt, W.pvt, W.hist, W.seg_s, W.seg_e, W.part, W.ml);
    BSA_STEP("fwd.slc",
             bsa::launch_slc1_fwd(D, q, k, v, valid, saved->sel_idx, S1, ob + ob_stride, lse + 2 * rows, st),
             "per-token selection attention");
  } else {
    BSA_STEP("fwd.slc",
             bsa::launch_slc_fwd(D, q, k, v, valid, saved->sel_idx, ob + ob_stride, lse + 2 * rows, st),
             "selection attention");
  }
  s = joiner.join();
  if (s != BSA_OK) return s;
  BSA_STEP("fwd.gate", bsa::launch_gate_fwd(D, ob, saved->o_cmp, gate, valid, o, st), "gate");
#undef BSA_STEP
  return BSA_OK;
}

bsa_status_t bsa_backward(const bsa_params_t* p, const void* q, const void* k, const void* v, const uint8_t* valid,
                          const float* gate, const bsa_mlp_t* phi_k, const bsa_mlp_t* phi_v, const bsa_mlp_t* phi_q,
                          const bsa_saved_t* saved, const void* d_o, float* dq, float* dk, float* dv, float* dgate,
                          const bsa_mlp_grad_t* dphi_k, const bsa_mlp_grad_t* dphi_v, const bsa_mlp_grad_t* dphi_q,
                          void* ws, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  bsa::Dims D;
  bsa_status_t s = check_params(p, &D);
  if (s != BSA_OK) return s;
  if (!q || !k || !v || !gate || !d_o || !dq || !dk || !dv || !dgate)
    return fail(BSA_ERR_INVALID_ARGUMENT, "q, k, v, gate, d_o, dq, dk, dv and dgate must be non-NULL");
  if (!saved_ok(saved, D)) return fail(BSA_ERR_INVALID_ARGUMENT, "every saved buffer must be non-NULL");
  auto fullg = [](const bsa_mlp_grad_t* m) { return m && m->w1 && m->b1 && m->w2 && m->b2; };
  if (D.pool == 0 && (!mlp_ok(phi_k) || !mlp_ok(phi_v) || !fullg(dphi_k) || !fullg(dphi_v)))
    return fail(BSA_ERR_INVALID_ARGUMENT, "MLP pooling needs phi_k, phi_v, dphi_k and dphi_v with all four tensors");
  const bool q_grad = D.gcmp && D.qc_mlp;   // phi_q gets a gradient only through Eq. 15
  if (q_grad && (!mlp_ok(phi_q) || !fullg(dphi_q)))
    return fail(BSA_ERR_INVALID_ARGUMENT, "group compression with MLP coarsening needs phi_q and dphi_q");
  const BwdWs W = bwd_ws_layout(D);
  if (!ws || ws_bytes < W.total)
    return fail(BSA_ERR_WORKSPACE_TOO_SMALL, "backward workspace needs " + std::to_string(W.total) + " bytes");
  hipStream_t st = (hipStream_t)stream;
  std::lock_guard<std::mutex> lock(g_aux_mu);
  Aux aux;
  s = get_aux(&aux);
  if (s != BSA_OK) return s;
  if (g_streams < 2) aux.s = st;
  char* w = (char*)ws;
  bsa::BwdArgs A{};
  A.q = q; A.k = k; A.v = v; A.dout = d_o; A.valid = valid; A.gate = gate;
  A.o_branch = saved->o_branch; A.o_cmp = saved->o_cmp; A.lse = saved->lse; A.kcmp = saved->kcmp; A.vcmp = saved->vcmp;
  A.hid_k = saved->hid_k; A.hid_v = saved->hid_v; A.sel = saved->sel_idx; A.cvalid = saved->cvalid;
  A.dq = dq; A.dk = dk; A.dv = dv; A.dgate = dgate;
  A.R = (float*)(w + W.R);
  A.terms = (float*)(w + W.terms);
  A.kc_lp = w + W.kc_lp; A.vc_lp = w + W.vc_lp;
  A.dkc_part = (float*)(w + W.dkc_part); A.dvc_part = (float*)(w + W.dvc_part);
  A.dkc = (float*)(w + W.dkc); A.dvc = (float*)(w + W.dvc);
  A.pair_keys = (uint32_t*)(w + W.pk); A.pair_vals = (uint32_t*)(w + W.pv);
  A.pair_keys_tmp = (uint32_t*)(w + W.pkt); A.pair_vals_tmp = (uint32_t*)(w + W.pvt);
  A.sort_hist = (uint32_t*)(w + W.hist);
  A.seg_start = (int*)(w + W.seg_s); A.seg_end = (int*)(w + W.seg_e);
  A.qcmp = saved->qcmp; A.ocmp = saved->ocmp; A.qc_lp = w + W.qc_lp; A.doc = w + W.doc; A.t4c = (float*)(w + W.t4c);
  A.dqc = (float*)(w + W.dqc);
  A.lse_ws = (float*)(w + W.lse);
  A.lsec_ws = (float*)(w + W.lsec);
  if (D.g == 1)
    A.s1 = slc1_ws(D, w, W.pk, W.pv, W.pkt, W.pvt, W.hist, W.seg_s, W.seg_e, W.dqpart, D.store_lse ? (size_t)-1 : W.ml);
  // Schedule over the two streams (with one stream the same order runs on `st`): the row
  // terms and the ball and compressed dK/dV passes first, alone; then the dQ chain (ball
  // writes, compressed and selection add) on the auxiliary stream beside the MLP backward
  // and the selection dK/dV pass on the caller's. (Running the selection and MLP passes
  // beside the compressed dK/dV pass instead gave the same step time: the kernels do not
  // share CUs well, and the compressed pass's own time then includes the sharing.)
  AuxJoin joiner(aux, st);
  BSA_TRY(bsa::launch_bwd_stage(D, A, bsa::BwdStage::prep, st), "backward row terms");
  if (g_streams != 0) {
    BSA_TRY(bsa::launch_bwd_stage(D, A, bsa::BwdStage::kv_pair, st), "ball and compressed dK/dV");
  } else {
    BSA_TRY(bsa::launch_bwd_stage(D, A, bsa::BwdStage::kv_ball, st), "ball dK/dV");
    BSA_TRY(bsa::launch_bwd_stage(D, A, bsa::BwdStage::kv_cmp, st), "compressed dK/dV");
  }
  if (aux.s != st && (hipEventRecord(aux.fork, st) != hipSuccess || hipStreamWaitEvent(aux.s, aux.fork, 0) != hipSuccess))
    return fail(BSA_ERR_HIP, "forking the auxiliary stream failed");
  BSA_TRY(bsa::launch_bwd_stage(D, A, bsa::BwdStage::dq_ball, aux.s), "ball dQ");
  BSA_TRY(bsa::launch_bwd_stage(D, A, bsa::BwdStage::dq_cmp, aux.s), "compressed dQ");
  if (D.g != 1) BSA_TRY(bsa::launch_bwd_stage(D, A, bsa::BwdStage::dq_slc, aux.s), "selection dQ");
  bsa::MlpBwdWs mw{(float*)(w + W.dpre), (float*)(w + W.pw1), (float*)(w + W.psm), (void*)(w + W.w1lp),
                   W.mlp_chunks, W.mlp_chunks_small, (void*)(w + W.dplp)};
  bsa::Mlp mk{}, mv{};
  bsa::MlpGrad gk{}, gv{};
  if (D.pool == 0) {
    mk = {phi_k->w1, phi_k->b1, phi_k->w2, phi_k->b2};
    mv = {phi_v->w1, phi_v->b1, phi_v->w2, phi_v->b2};
    gk = {dphi_k->w1, dphi_k->b1, dphi_k->w2, dphi_k->b2};
    gv = {dphi_v->w1, dphi_v->b1, dphi_v->w2, dphi_v->b2};
  }
  hipError_t e;
  BSA_PHASE("bwd.mlp", st, e = bsa::launch_compress_bwd(D, k, valid, mk, saved->hid_k, A.dkc, dk, gk, mw, st));
  BSA_TRY(e, "compression backward K");
  BSA_PHASE("bwd.mlp", st, e = bsa::launch_compress_bwd(D, v, valid, mv, saved->hid_v, A.dvc, dv, gv, mw, st));
  BSA_TRY(e, "compression backward V");
  const bsa::Slc1Ws S1 = slc1_ws(D, w, W.pk, W.pv, W.pkt, W.pvt, W.hist, W.seg_s, W.seg_e, W.dqpart, (size_t)-1);
  if (D.g == 1) {
    BSA_TRY(bsa::launch_slc1_bwd(D, q, k, v, d_o, valid, saved->sel_idx, (const float4*)A.terms + 2 * D.rows(), S1,
                                 dk, dv, st),
            "per-token selection backward");
  } else {
    const uint32_t* slc_groups = nullptr;
    BSA_TRY(bsa::launch_slc_csr(D, A, st, &slc_groups), "selection lists");
    BSA_TRY(bsa::launch_slc_kv(D, A, slc_groups, st), "selection dK/dV");
  }
  s = joiner.join();
  if (s != BSA_OK) return s;
  if (D.g == 1) {   // the dQ parts of the per-token selection, after the dQ chain
    BSA_PHASE("bwd.dq_slc", st, e = bsa::launch_slc1_merge_dq(D, saved->sel_idx, valid, S1, dq, st));
    BSA_TRY(e, "per-token selection dQ");
  }
  if (D.gcmp) {
    // coarse-query gradient of Eq. 15 through phi_q (or the block mean) into dQ
    bsa::Dims Dq = D;
    Dq.pool = D.qc_mlp ? 0 : 1;
    bsa::Mlp mq{};
    bsa::MlpGrad gq{};
    if (q_grad) {
      mq = {phi_q->w1, phi_q->b1, phi_q->w2, phi_q->b2};
      gq = {dphi_q->w1, dphi_q->b1, dphi_q->w2, dphi_q->b2};
    }
    BSA_PHASE("bwd.mlp", st, e = bsa::launch_compress_bwd(Dq, q, valid, mq, saved->hid_q, A.dqc, dq, gq, mw, st));
    BSA_TRY(e, "query coarsening backward");
  }
  return BSA_OK;
}

}  // extern "C"

// ---- the transformer block around the layer (Section 3.1) ----

namespace {

struct BlockDims {
  bsa::Dims D;
  int C, F;
  long long M;   // token rows B * N
};

bsa_status_t check_block(const bsa_params_t* p, int32_t ffn, BlockDims* X) {
  bsa_status_t s = check_params(p, &X->D);
  if (s != BSA_OK) return s;
  const bsa::Dims& D = X->D;
  if (!D.bf16) return fail(BSA_ERR_UNSUPPORTED, "the block runs bf16 layers only");
  X->C = D.H * D.d;
  if (X->C != 128 && X->C != 256 && X->C != 512 && X->C != 1024)
    return fail(BSA_ERR_UNSUPPORTED, "the block needs heads * head_dim in {128, 256, 512, 1024}");
  if (ffn <= 0 || ffn % 128 != 0) return fail(BSA_ERR_UNSUPPORTED, "ffn_dim must be a positive multiple of 128");
  X->F = ffn;
  X->M = (long long)D.B * D.N;
  if (X->M > (1LL << 30) || X->M * 2 * ffn >= (1LL << 40))
    return fail(BSA_ERR_UNSUPPORTED, "batch * n (or its SwiGLU activations) too large");
  return BSA_OK;
}

struct BlockSavedLayout {
  size_t layer, r1, r2, xn1, gate, q, k, v, o, h, xn2, uw, a, total;
};

BlockSavedLayout block_saved_layout(const BlockDims& X) {
  BlockSavedLayout L{};
  const size_t M = (size_t)X.M, C = (size_t)X.C, F = (size_t)X.F;
  size_t off = 0;
  auto put = [&](size_t bytes) { size_t o = off; off += align256(bytes); return o; };
  L.layer = put(saved_layout(X.D).total);
  L.r1 = put(4 * M);
  L.r2 = put(4 * M);
  L.xn1 = put(2 * M * C);
  L.gate = put(4 * 3 * M);
  L.q = put(2 * M * C);
  L.k = put(2 * M * C);
  L.v = put(2 * M * C);
  L.o = put(2 * M * C);
  L.h = put(4 * M * C);
  L.xn2 = put(2 * M * C);
  L.uw = put(2 * M * 2 * F);
  L.a = put(2 * M * F);
  L.total = off;
  return L;
}

struct BlockFwdWs {
  size_t wqkv, wo, w13, w2, layer, total;
};

BlockFwdWs block_fwd_ws(const BlockDims& X) {
  BlockFwdWs L{};
  const size_t C = (size_t)X.C, F = (size_t)X.F;
  size_t off = 0;
  auto put = [&](size_t bytes) { size_t o = off; off += align256(bytes); return o; };
  L.wqkv = put(2 * 3 * C * C);
  L.wo = put(2 * C * C);
  L.w13 = put(2 * 2 * F * C);
  L.w2 = put(2 * C * F);
  L.layer = put(fwd_ws_layout(X.D).total);
  L.total = off;
  return L;
}

// weight-gradient products: dW [Mo, No] = sum over the M tokens; split-K partials
struct WgradShape {
  int Mo, No;
};

size_t wgrad_part_bytes(const BlockDims& X) {
  const WgradShape sh[4] = {{X.C, X.F}, {2 * X.F, X.C}, {X.C, X.C}, {3 * X.C, X.C}};
  size_t best = 0;
  for (const WgradShape& w : sh) {
    const size_t b = sizeof(float) * (size_t)bsa::gemm_splits(w.Mo, w.No, X.M) * w.Mo * w.No;
    best = b > best ? b : best;
  }
  return best;
}

struct BlockBwdWs {
  size_t wqkvt, wot, w13t, w2t, dy16, part, duw, dxn, dh, dh16, do16, dq, dk, dv, dgate, dqkv, npart, layer,
      total;
};

BlockBwdWs block_bwd_ws(const BlockDims& X) {
  BlockBwdWs L{};
  const size_t M = (size_t)X.M, C = (size_t)X.C, F = (size_t)X.F;
  size_t off = 0;
  auto put = [&](size_t bytes) { size_t o = off; off += align256(bytes); return o; };
  L.wqkvt = put(2 * 3 * C * C);
  L.wot = put(2 * C * C);
  L.w13t = put(2 * 2 * F * C);
  L.w2t = put(2 * C * F);
  L.dy16 = put(2 * M * C);
  L.part = put(wgrad_part_bytes(X));
  L.duw = put(2 * M * 2 * F);
  L.dxn = put(4 * M * C);
  L.dh = put(4 * M * C);
  L.dh16 = put(2 * M * C);
  L.do16 = put(2 * M * C);
  L.dq = put(4 * M * C);
  L.dk = put(4 * M * C);
  L.dv = put(4 * M * C);
  L.dgate = put(4 * 3 * M);
  L.dqkv = put(2 * M * 3 * C);
  L.npart = put(bsa::rmsnorm_bwd_part_bytes(X.M, X.C));
  L.layer = put(bwd_ws_layout(X.D).total);
  L.total = off;
  return L;
}

int ilog2(long long x) {
  int r = 0;
  while ((1LL << r) < x) ++r;
  return r;
}

bsa::GemmMat plain(const void* p, long long ld) { return bsa::GemmMat{(const uint16_t*)p, ld, 0, 0, 0}; }

bsa::GemmMat heads_mat(const BlockDims& X, const void* p) {
  return bsa::GemmMat{(const uint16_t*)p, 0, X.D.H, ilog2(X.D.N), ilog2(X.D.d)};
}

bsa::GemmOut out_f32(float* out, long long ldc, const float* res = nullptr, long long ldr = 0) {
  bsa::GemmOut o{};
  o.epi = bsa::kEpiF32;
  o.out = out;
  o.ldc = ldc;
  o.res = res;
  o.ldr = ldr;
  return o;
}

bsa::GemmOut out_heads(const BlockDims& X, void* p0, void* p1, void* p2) {
  bsa::GemmOut o{};
  o.epi = bsa::kEpiHeads;
  o.parts[0] = (uint16_t*)p0;
  o.parts[1] = (uint16_t*)p1;
  o.parts[2] = (uint16_t*)p2;
  o.part_cols = X.C;
  o.heads = X.D.H;
  o.lgn = ilog2(X.D.N);
  o.lgd = ilog2(X.D.d);
  return o;
}

// dW [Mo, No] = A^T B over the M token rows (A [M, Mo], B [M, No]) into out (rows < split_row)
// and out2 (the remaining rows, when out2 is given).
hipError_t wgrad(const BlockDims& X, const bsa::GemmMat& a, const bsa::GemmMat& b, int Mo, int No, float* part,
                 float* out, float* out2, int split_row, hipStream_t st) {
  const int S = bsa::gemm_splits(Mo, No, X.M);
  bsa::GemmOut o{};
  o.epi = bsa::kEpiPart;
  o.out = part;
  o.ldc = No;
  hipError_t e = bsa::launch_gemm(true, a, b, Mo, No, X.M, S, o, st);
  if (e != hipSuccess) return e;
  const long long stride = (long long)Mo * No;
  if (!out2) return bsa::launch_splitk_sum(part, S, stride, stride, out, st);
  e = bsa::launch_splitk_sum(part, S, stride, (long long)split_row * No, out, st);
  if (e != hipSuccess) return e;
  return bsa::launch_splitk_sum(part + (long long)split_row * No, S, stride, (long long)(Mo - split_row) * No, out2,
                                st);
}

bool mlp_ok(const bsa_mlp_t& m) { return m.w1 && m.b1 && m.w2 && m.b2; }

}  // namespace

#define BSA_HIP(expr, where) BSA_TRY((expr), (where))

extern "C" {

bsa_status_t bsa_block_sizes(const bsa_params_t* p, int32_t ffn_dim, size_t* ws_fwd_bytes, size_t* ws_bwd_bytes,
                             size_t* saved_bytes) {
  g_last_error.clear();
  BlockDims X;
  bsa_status_t s = check_block(p, ffn_dim, &X);
  if (s != BSA_OK) return s;
  if (ws_fwd_bytes) *ws_fwd_bytes = block_fwd_ws(X).total;
  if (ws_bwd_bytes) *ws_bwd_bytes = block_bwd_ws(X).total;
  if (saved_bytes) *saved_bytes = block_saved_layout(X).total;
  return BSA_OK;
}

bsa_status_t bsa_block_saved_view(const bsa_params_t* p, int32_t ffn_dim, void* base, bsa_block_saved_t* out) {
  g_last_error.clear();
  BlockDims X;
  bsa_status_t s = check_block(p, ffn_dim, &X);
  if (s != BSA_OK) return s;
  if (!base || !out) return fail(BSA_ERR_INVALID_ARGUMENT, "base and out must be non-NULL");
  const BlockSavedLayout L = block_saved_layout(X);
  char* c = (char*)base;
  s = bsa_saved_view(p, c + L.layer, &out->layer);
  if (s != BSA_OK) return s;
  out->rstd1 = (float*)(c + L.r1);
  out->rstd2 = (float*)(c + L.r2);
  out->xn1 = c + L.xn1;
  out->gate = (float*)(c + L.gate);
  out->q = c + L.q;
  out->k = c + L.k;
  out->v = c + L.v;
  out->o = c + L.o;
  out->h = (float*)(c + L.h);
  out->xn2 = c + L.xn2;
  out->uw = c + L.uw;
  out->a = c + L.a;
  return BSA_OK;
}

bsa_status_t bsa_block_forward(const bsa_params_t* p, int32_t ffn_dim, const bsa_block_weights_t* w, const float* x,
                               const uint8_t* valid, float* y, const bsa_block_saved_t* saved, void* ws,
                               size_t ws_bytes, void* stream) {
  g_last_error.clear();
  BlockDims X;
  bsa_status_t s = check_block(p, ffn_dim, &X);
  if (s != BSA_OK) return s;
  if (!w || !x || !y || !saved || !ws) return fail(BSA_ERR_INVALID_ARGUMENT, "w, x, y, saved and ws must be non-NULL");
  if (!w->g1 || !w->wqkv || !w->wg || !w->wo || !w->g2 || !w->w1 || !w->w3 || !w->w2)
    return fail(BSA_ERR_INVALID_ARGUMENT, "every block weight must be non-NULL");
  if (x == y) return fail(BSA_ERR_INVALID_ARGUMENT, "y may not alias x");
  const BlockFwdWs L = block_fwd_ws(X);
  if (ws_bytes < L.total) return fail(BSA_ERR_WORKSPACE_TOO_SMALL, "block forward workspace too small");
  const bsa_block_saved_t& sv = *saved;
  if (!sv.rstd1 || !sv.rstd2 || !sv.xn1 || !sv.gate || !sv.q || !sv.k || !sv.v || !sv.o || !sv.h || !sv.xn2 || !sv.uw ||
      !sv.a)
    return fail(BSA_ERR_INVALID_ARGUMENT, "saved tensors must be non-NULL");
  hipStream_t st = (hipStream_t)stream;
  const int C = X.C, F = X.F;
  const long long M = X.M;
  char* c = (char*)ws;
  uint16_t *wqkv = (uint16_t*)(c + L.wqkv), *wo = (uint16_t*)(c + L.wo), *w13 = (uint16_t*)(c + L.w13),
           *w2 = (uint16_t*)(c + L.w2);
  BSA_PHASE("blk.elem", st, {
    BSA_HIP(bsa::launch_cast_bf16(w->wqkv, 3LL * C * C, wqkv, st), "cast wqkv");
    BSA_HIP(bsa::launch_cast_bf16(w->wo, (long long)C * C, wo, st), "cast wo");
    BSA_HIP(bsa::launch_cast_w13(w->w1, w->w3, F, C, bsa::gemm_wave_cols((int)M, 2 * F), w13, st), "cast w1, w3");
    BSA_HIP(bsa::launch_cast_bf16(w->w2, (long long)C * F, w2, st), "cast w2");
  });
  BSA_PHASE("blk.norm", st,
            BSA_HIP(bsa::launch_rmsnorm_fwd(x, w->g1, w->wg, M, C, (uint16_t*)sv.xn1, sv.rstd1, sv.gate, st),
                    "rmsnorm 1"));
  BSA_PHASE("blk.gemm", st,
            BSA_HIP(bsa::launch_gemm(false, plain(sv.xn1, C), plain(wqkv, C), (int)M, 3 * C, C, 1,
                                     out_heads(X, sv.q, sv.k, sv.v), st),
                    "qkv product"));
  s = bsa_forward(p, sv.q, sv.k, sv.v, valid, sv.gate, &w->phi_k, &w->phi_v, mlp_ok(w->phi_q) ? &w->phi_q : nullptr,
                  sv.o, &sv.layer, c + L.layer, L.total - L.layer, stream);
  if (s != BSA_OK) return s;
  BSA_PHASE("blk.gemm", st,
            BSA_HIP(bsa::launch_gemm(false, heads_mat(X, sv.o), plain(wo, C), (int)M, C, C, 1, out_f32(sv.h, C, x, C),
                                     st),
                    "output projection"));
  BSA_PHASE("blk.norm", st,
            BSA_HIP(bsa::launch_rmsnorm_fwd(sv.h, w->g2, nullptr, M, C, (uint16_t*)sv.xn2, sv.rstd2, nullptr, st),
                    "rmsnorm 2"));
  BSA_PHASE("blk.gemm", st, {
    bsa::GemmOut o{};
    o.epi = bsa::kEpiSwigluFwd;
    o.out = sv.uw;
    o.out2 = sv.a;
    o.ffn = F;
    BSA_HIP(bsa::launch_gemm(false, plain(sv.xn2, C), plain(w13, C), (int)M, 2 * F, C, 1, o, st), "swiglu");
  });
  BSA_PHASE("blk.gemm", st,
            BSA_HIP(bsa::launch_gemm(false, plain(sv.a, F), plain(w2, F), (int)M, C, F, 1, out_f32(y, C, sv.h, C), st),
                    "swiglu out"));
  return BSA_OK;
}

bsa_status_t bsa_block_backward(const bsa_params_t* p, int32_t ffn_dim, const bsa_block_weights_t* w, const float* x,
                                const uint8_t* valid, const bsa_block_saved_t* saved, const float* dy, float* dx,
                                const bsa_block_grads_t* dw, void* ws, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  BlockDims X;
  bsa_status_t s = check_block(p, ffn_dim, &X);
  if (s != BSA_OK) return s;
  if (!w || !x || !saved || !dy || !dx || !dw || !ws)
    return fail(BSA_ERR_INVALID_ARGUMENT, "w, x, saved, dy, dx, dw and ws must be non-NULL");
  if (!w->g1 || !w->wqkv || !w->wg || !w->wo || !w->g2 || !w->w1 || !w->w3 || !w->w2)
    return fail(BSA_ERR_INVALID_ARGUMENT, "every block weight must be non-NULL");
  if (!dw->g1 || !dw->wqkv || !dw->wg || !dw->wo || !dw->g2 || !dw->w1 || !dw->w3 || !dw->w2)
    return fail(BSA_ERR_INVALID_ARGUMENT, "every block weight gradient must be non-NULL");
  const BlockBwdWs L = block_bwd_ws(X);
  if (ws_bytes < L.total) return fail(BSA_ERR_WORKSPACE_TOO_SMALL, "block backward workspace too small");
  const bsa_block_saved_t& sv = *saved;
  hipStream_t st = (hipStream_t)stream;
  const int C = X.C, F = X.F;
  const long long M = X.M;
  char* c = (char*)ws;
  auto u16 = [&](size_t off) { return (uint16_t*)(c + off); };
  auto f32 = [&](size_t off) { return (float*)(c + off); };
  uint16_t *wqkvt = u16(L.wqkvt), *wot = u16(L.wot), *w13t = u16(L.w13t), *w2t = u16(L.w2t);
  uint16_t *dy16 = u16(L.dy16), *duw = u16(L.duw), *dh16 = u16(L.dh16), *do16 = u16(L.do16), *dqkv = u16(L.dqkv);
  float *part = f32(L.part), *dxn = f32(L.dxn), *dh = f32(L.dh), *dq = f32(L.dq), *dk = f32(L.dk),
        *dv = f32(L.dv), *dgate = f32(L.dgate), *npart = f32(L.npart);
  BSA_PHASE("blk.elem", st, {
    BSA_HIP(bsa::launch_cast_t(w->wqkv, 3 * C, C, wqkvt, 3 * C, st), "cast wqkv^T");
    BSA_HIP(bsa::launch_cast_t(w->wo, C, C, wot, C, st), "cast wo^T");
    BSA_HIP(bsa::launch_cast_t(w->w1, F, C, w13t, 2 * F, st), "cast w1^T");
    BSA_HIP(bsa::launch_cast_t(w->w3, F, C, w13t + F, 2 * F, st), "cast w3^T");
    BSA_HIP(bsa::launch_cast_t(w->w2, C, F, w2t, C, st), "cast w2^T");
    BSA_HIP(bsa::launch_cast_bf16(dy, M * C, dy16, st), "cast dy");
  });
  // SwiGLU sublayer
  BSA_PHASE("blk.wgrad", st,
            BSA_HIP(wgrad(X, plain(dy16, C), plain(sv.a, F), C, F, part, dw->w2, nullptr, 0, st), "dW2"));
  BSA_PHASE("blk.gemm", st, {
    bsa::GemmOut o{};
    o.epi = bsa::kEpiSwigluBwd;
    o.out = duw;
    o.aux = (const uint16_t*)sv.uw;
    o.ffn = F;
    BSA_HIP(bsa::launch_gemm(false, plain(dy16, C), plain(w2t, C), (int)M, F, C, 1, o, st), "swiglu bwd");
  });
  BSA_PHASE("blk.wgrad", st,
            BSA_HIP(wgrad(X, plain(duw, 2 * F), plain(sv.xn2, C), 2 * F, C, part, dw->w1, dw->w3, F, st), "dW13"));
  BSA_PHASE("blk.gemm", st,
            BSA_HIP(bsa::launch_gemm(false, plain(duw, 2 * F), plain(w13t, 2 * F), (int)M, C, 2 * F, 1,
                                     out_f32(dxn, C), st),
                    "dxn2"));
  BSA_PHASE("blk.norm", st,
            BSA_HIP(bsa::launch_rmsnorm_bwd(dxn, sv.h, sv.rstd2, w->g2, dy, nullptr, nullptr, M, C, dh, dh16, npart,
                                            dw->g2, nullptr, st),
                    "rmsnorm 2 bwd"));
  // attention sublayer
  BSA_PHASE("blk.wgrad", st,
            BSA_HIP(wgrad(X, plain(dh16, C), heads_mat(X, sv.o), C, C, part, dw->wo, nullptr, 0, st), "dWo"));
  BSA_PHASE("blk.gemm", st,
            BSA_HIP(bsa::launch_gemm(false, plain(dh16, C), plain(wot, C), (int)M, C, C, 1,
                                     out_heads(X, do16, nullptr, nullptr), st),
                    "dO"));
  const bool dq_mlp = X.D.qc_mlp && X.D.gcmp;
  s = bsa_backward(p, sv.q, sv.k, sv.v, valid, sv.gate, &w->phi_k, &w->phi_v, mlp_ok(w->phi_q) ? &w->phi_q : nullptr,
                   &sv.layer, do16, dq, dk, dv, dgate, &dw->phi_k, &dw->phi_v, dq_mlp ? &dw->phi_q : nullptr,
                   c + L.layer, L.total - L.layer, stream);
  if (s != BSA_OK) return s;
  BSA_PHASE("blk.elem", st,
            BSA_HIP(bsa::launch_pack_qkv(dq, dk, dv, M, C, X.D.H, ilog2(X.D.N), ilog2(X.D.d), dqkv, st), "pack dqkv"));
  BSA_PHASE("blk.wgrad", st,
            BSA_HIP(wgrad(X, plain(dqkv, 3 * C), plain(sv.xn1, C), 3 * C, C, part, dw->wqkv, nullptr, 0, st),
                    "dWqkv"));
  BSA_PHASE("blk.gemm", st,
            BSA_HIP(bsa::launch_gemm(false, plain(dqkv, 3 * C), plain(wqkvt, 3 * C), (int)M, C, 3 * C, 1,
                                     out_f32(dxn, C), st),
                    "dxn1"));
  BSA_PHASE("blk.norm", st,
            BSA_HIP(bsa::launch_rmsnorm_bwd(dxn, x, sv.rstd1, w->g1, dh, dgate, w->wg, M, C, dx, nullptr, npart,
                                            dw->g1, dw->wg, st),
                    "rmsnorm 1 bwd"));
  return BSA_OK;
}

}  // extern "C"
