// Host-side launchers of the BSA kernels (internal to the library).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace bsa {

// Layer sizes after validation (notation of Section 2).
struct Dims {
  int B, H, N, d;      // clouds, heads, token slots, head dim
  int m;               // ball size
  int l;               // compression block (= stride)
  int ls;              // selection block
  int k;               // top-k
  int g;               // query group size
  int mask_own;        // exclude own-ball blocks from selection
  int pool;            // 0 = MLP, 1 = mean
  int bf16;            // 1 = bf16 storage of Q/K/V/O, 0 = f32
  int qc_mlp;          // coarse queries by the MLP phi_q over blocks of l (Eq. 13)
  int gcmp;            // group compression (Eq. 15)
  int store_lse;       // 1: the forward keeps the log-sum-exp rows; 0: the backward recomputes them
  float scale;         // softmax scale
  long long rows() const { return (long long)B * H * N; }
  // coarse queries come from blocks of l (Eq. 13), not the group mean computed by the top-k
  bool block_coarse() const { return qc_mlp || gcmp; }
  long long cmp_rows() const { return (long long)B * H * (N / l); }
};

struct Mlp { const float *w1, *b1, *w2, *b2; };
struct MlpGrad { float *w1, *b1, *w2, *b2; };

// tree.hip
size_t tree_workspace_bytes(int64_t n_real, int64_t n_pad, int batch);
// The allocation-free tree build's static scratch: its slot limit (batch * n_pad), its size,
// and its address on the current device (looked up once per device).
int64_t tree_scratch_slots();
size_t tree_scratch_bytes();
hipError_t tree_scratch(void** ptr);
hipError_t launch_build_tree(const float* pts, int64_t n_real, int dim, int64_t n_pad, int batch,
                             int* perm, void* ws, hipStream_t st);
hipError_t launch_permute(const void* src, const int* perm, int64_t n_real, int64_t n_pad, int batch,
                          int heads, int hd, int dtype, void* dst, uint8_t* valid, bool inverse,
                          hipStream_t st);

// compress.hip: compression phi of Eq. 5 and its backward
hipError_t launch_block_valid(const Dims& D, const uint8_t* valid, uint8_t* cvalid, hipStream_t st);
// One compression: x [B, H, N, d] in the storage type; out (float32) and out_lp (the rows in
// the storage type, multiplied by lp_scale: the compressed keys of bf16 layers carry the
// softmax scale times log2(e) there; see launch_cmp_fwd) are [B, H, N/l, d]; pre: the MLP's
// pre-activations (unused for mean pooling); w1t_ws: l*d*d elements of workspace.
struct CompressJob {
  const void* x;
  Mlp phi;
  float* out;
  float* pre;
  void* out_lp;
  void* w1t_ws;
  float lp_scale;
};
// n = 1 or 2 compressions of the same shape (the keys and values share one launch)
hipError_t launch_compress_fwd(const Dims& D, const CompressJob* jobs, int n, const uint8_t* valid, hipStream_t st);
// the bf16 layers' scale of the compressed keys' storage-type copy
inline float cmp_key_scale(const Dims& D) { return D.bf16 ? D.scale * 1.4426950408889634f : 1.0f; }

// select.hip: pooled-query block scores and group top-k (Eq. 6, 7, 10-12, 14)
// qpool: B*H*(N/g)*d floats of coarse queries; written here (group mean of Eq. 11) unless
// `given`, when it already holds them (Eq. 13); kplanes: 3 * B*H*(N/l)*d bf16 of workspace
// (the compressed keys in three bf16 parts)
hipError_t launch_select_topk(const Dims& D, const void* q, const uint8_t* valid, const float* kcmp,
                              const uint8_t* cvalid, int* sel, float* qpool, bool given, uint16_t* kplanes,
                              hipStream_t st);

// attn_fwd.hip: the three attention branches (Eq. 3, 5, 8) and the gate (Eq. 9)
hipError_t launch_ball_fwd(const Dims& D, const void* q, const void* k, const void* v, const uint8_t* valid,
                           void* o, float* lse, hipStream_t st);
// the compressed branch writes float32 rows (its backward forms the softmax delta from them)
hipError_t launch_cmp_fwd(const Dims& D, const void* q, const void* kc, const void* vc, const uint8_t* valid,
                          const uint8_t* cvalid, float* o, float* lse, hipStream_t st);
hipError_t launch_slc_fwd(const Dims& D, const void* q, const void* k, const void* v, const uint8_t* valid,
                          const int* sel, void* o, float* lse, hipStream_t st);
// both in one launch for unmasked bf16 layers (call only where ball_cmp_fwd_fits and
// there is no validity mask; else hipErrorNotSupported): ob and lse_ball as for
// launch_ball_fwd, ocmp and lse_cmp as for launch_cmp_fwd
bool ball_cmp_fwd_fits(const Dims& D);
hipError_t launch_ball_cmp_fwd(const Dims& D, const void* q, const void* k, const void* v, const void* kc, const void* vc,
                               void* ob, float* lse_ball, float* ocmp, float* lse_cmp, hipStream_t st);
// group compression (Eq. 15): coarse attention [B, H, N/l, d] (float32 outputs) and its
// copy to the token rows (float32)
hipError_t launch_cmp_coarse_fwd(const Dims& D, const void* qc, const void* kc, const void* vc, const uint8_t* cvalid,
                                 float* oc, float* lsec, hipStream_t st);
hipError_t launch_expand_coarse(const Dims& D, const float* oc, const float* lsec, const uint8_t* valid, float* ocmp,
                                float* lse, hipStream_t st);
// ob: ball and selection outputs [2, B, H, N, d] (storage type); ocmp: the compressed
// branch's [B, H, N, d] float32
hipError_t launch_gate_fwd(const Dims& D, const void* ob, const float* ocmp, const float* gate, const uint8_t* valid,
                           void* o, hipStream_t st);

// Buffers of the per-token selection (g = 1, slc_token.hip), block-major.
struct Slc1Ws {
  uint32_t *keys, *vals, *keys_tmp, *vals_tmp, *hist;   // (query, slot) pairs and their sort
  int *seg_start, *seg_end;                             // [B*H*N/l'] pair range of each block
  float* part;   // [pairs, d] forward: unnormalised partial outputs; backward: dQ parts
  float* ml;     // [pairs, 2] forward: scaled max and sum of each partial softmax
};

// Backward pass buffers (inputs, saved tensors, outputs and workspace parts).
struct BwdArgs {
  const void *q, *k, *v, *dout;
  const uint8_t* valid;
  const float* gate;
  const void* o_branch;          // [2, B, H, N, d] ball and selection outputs (storage type)
  const float* o_cmp;            // [B, H, N, d] compressed-branch output (float32)
  const float *lse, *kcmp, *vcmp, *hid_k, *hid_v;
  const int* sel;
  const uint8_t* cvalid;
  float *dq, *dk, *dv, *dgate;
  // workspace
  float* R;                      // [3, B, H, N]
  float* terms;                  // [3, B, H, N, 4]: log2 LSE, s, s * R, 0 per query row
  void *kc_lp, *vc_lp;           // compressed tokens in the storage type
  float *dkc_part, *dvc_part;    // [chunks, B, H, N/l, d]
  float *dkc, *dvc;              // [B, H, N/l, d]
  uint32_t *pair_keys, *pair_vals, *pair_keys_tmp, *pair_vals_tmp, *sort_hist;
  // group compression (Eq. 15)
  const float* qcmp;             // [B, H, N/l, d] coarse queries
  const float* ocmp;             // [B, H, N/l, d] their attention outputs (float32)
  void* qc_lp;                   // coarse queries in the storage type
  void* doc;                     // [B, H, N/l, d] dO of the coarse queries, storage type
  float* t4c;                    // [B, H, N/l] packed row terms of the coarse queries
  float* dqc;                    // [B, H, N/l, d] gradient of the coarse queries
  int *seg_start, *seg_end;
  const uint32_t* pair_groups;   // set internally: sorted group ids
  // store_lse = 0: the log-sum-exp rows are recomputed into lse_ws before the first pass
  float* lse_ws;                 // [3, B, H, N]
  float* lsec_ws;                // [B, H, N/l] coarse rows (group compression)
  Slc1Ws s1;                     // per-token selection buffers (g = 1; ml holds 2 floats per pair)
};

// attn_bwd.hip: the backward pass in stages. What each stage reads and writes:
//   prep     casts K^/V^ (and the coarse queries) to the storage type; recomputes the LSE
//            rows if not stored; writes R, the packed row terms and dgate (and the coarse
//            queries' dO and terms under group compression). Every later stage needs it.
//   kv_ball  writes dK, dV (the first writer of both).
//   kv_cmp   writes dK^, dV^ (dkc, dvc).
//   kv_pair  kv_ball and kv_cmp (one launch for unmasked bf16 layers, else the two).
//   dq_ball  writes dQ (the first writer).
//   dq_cmp   adds into dQ (group compression: writes the coarse-query gradient instead).
//   dq_slc   adds into dQ (g >= 8).
// launch_slc_csr inverts the selection lists (no dependency but prep); launch_slc_kv adds
// into dK, dV; launch_compress_bwd (compress.hip) adds dK^/dV^'s token gradients into dK,
// dV. Stages that add into the same tensor must be ordered after its first writer and
// after each other.
enum class BwdStage { prep, kv_ball, kv_cmp, kv_pair, dq_ball, dq_cmp, dq_slc };
hipError_t launch_bwd_stage(const Dims& D, const BwdArgs& A, BwdStage stage, hipStream_t st);
hipError_t launch_slc_csr(const Dims& D, const BwdArgs& A, hipStream_t st, const uint32_t** groups_out);
hipError_t launch_slc_kv(const Dims& D, const BwdArgs& A, const uint32_t* groups, hipStream_t st);

// compress.hip: backward of phi (dK^ -> token gradients added into dx, weight gradients)
struct MlpBwdWs {
  float* dpre;        // [rows, d]
  float* part_w1;     // [chunks, l*d, d]
  float* part_small;  // [chunks_small, d*d + 2d]
  void* w1_lp;        // [l*d, d] W1 in the storage type
  int chunks, chunks_small;
  void* dpre_lp;      // [rows, d] dpre in the storage type
};
int mlp_bwd_chunks(const Dims& D);
int mlp_bwd_chunks_small(const Dims& D);
hipError_t launch_compress_bwd(const Dims& D, const void* x, const uint8_t* valid, const Mlp& phi, const float* pre,
                               const float* dy, float* dx_accum, const MlpGrad& grad, const MlpBwdWs& ws,
                               hipStream_t st);

size_t slc1_pairs(const Dims& D);
hipError_t launch_slc1_csr(const Dims& D, const int* sel, const uint8_t* valid, const Slc1Ws& W, uint32_t** vals_out,
                           hipStream_t st);
hipError_t launch_slc1_fwd(const Dims& D, const void* q, const void* k, const void* v, const uint8_t* valid,
                           const int* sel, const Slc1Ws& W, void* o, float* lse, hipStream_t st);
hipError_t launch_slc1_bwd(const Dims& D, const void* q, const void* k, const void* v, const void* dout,
                           const uint8_t* valid, const int* sel, const float4* t4, const Slc1Ws& W, float* dk,
                           float* dv, hipStream_t st);
hipError_t launch_slc1_merge_dq(const Dims& D, const int* sel, const uint8_t* valid, const Slc1Ws& W, float* dq,
                                hipStream_t st);

// tree.hip: stable LSD radix sort of (key, value) pairs on the low `bits` key bits.
size_t radix_sort_hist_words(long long n);
hipError_t launch_radix_sort_pairs(uint32_t* keys, uint32_t* vals, uint32_t* keys_tmp, uint32_t* vals_tmp,
                                   uint32_t* hist, long long n, int bits, uint32_t** keys_out, uint32_t** vals_out,
                                   hipStream_t st);

// block.hip: the dense parts of the transformer block (RMSNorm, channel products, SwiGLU)
// A bf16 operand of the block's products: element (r, c) of a logical row-major matrix.
// heads == 0: at p[r * ld + c]. heads > 0: the head-major layout [B, heads, n, d] of a
// logical [B * n, heads * d] matrix (n = 2^lgn, d = 2^lgd).
struct GemmMat {
  const uint16_t* p;
  long long ld;
  int heads, lgn, lgd;
};
// kEpiSwigluFwd: B rows interleave W_1 and W_3 (launch_cast_w13); writes
//   u | w (bf16 [M, 2 ffn], stacked) to out and silu(u) w (bf16 [M, ffn]) to out2.
// kEpiSwigluBwd: the product is da [M, ffn]; with u | w from aux writes du | dw (bf16
//   [M, 2 ffn]) to out.
enum GemmEpi { kEpiF32 = 0, kEpiBf16 = 1, kEpiHeads = 2, kEpiPart = 3, kEpiSwigluFwd = 4, kEpiSwigluBwd = 5 };
struct GemmOut {
  int epi;
  void* out;            // kEpiF32 / kEpiBf16: [M, ldc]; kEpiPart: f32 [splits][M][ldc]
  long long ldc;
  const float* res;     // kEpiF32: added to the product (may be NULL)
  long long ldr;
  uint16_t* parts[3];   // kEpiHeads: column block p (part_cols wide) -> head-major parts[p]
  int part_cols, heads, lgn, lgd;
  const uint16_t* aux;  // kEpiSwigluBwd: u | w
  void* out2;           // kEpiSwigluFwd: silu(u) w
  int ffn;
};
// C[M, N] = sum_k A(m, k) B(n, k); trans = false: A [M, K], B [N, K]; trans = true: A [K, M],
// B [K, N]. M, N multiples of 128, K of 64; splits > 1 only with kEpiPart.
hipError_t launch_gemm(bool trans, const GemmMat& a, const GemmMat& b, int M, int N, long long K, int splits,
                       const GemmOut& o, hipStream_t st);
int gemm_splits(int M, int N, long long K);
hipError_t launch_rmsnorm_fwd(const float* x, const float* gain, const float* wg, long long rows, int C, uint16_t* xn,
                              float* rstd, float* gate, hipStream_t st);
hipError_t launch_rmsnorm_bwd(const float* dxn, const float* x, const float* rstd, const float* gain, const float* dres,
                              const float* dgate, const float* wg, long long rows, int C, float* dx, uint16_t* dx16,
                              float* part, float* dgain, float* dwg, hipStream_t st);
size_t rmsnorm_bwd_part_bytes(long long rows, int C);
hipError_t launch_splitk_sum(const float* part, int S, long long stride, long long count, float* out, hipStream_t st);
hipError_t launch_pack_qkv(const float* dq, const float* dk, const float* dv, long long rows, int C, int H, int lgn,
                           int lgd, uint16_t* out, hipStream_t st);
hipError_t launch_cast_bf16(const float* src, long long n, uint16_t* dst, hipStream_t st);
// [W_1; W_3] interleaved in groups of G rows for kEpiSwigluFwd; G = gemm_wave_cols(M, 2F)
hipError_t launch_cast_w13(const float* w1, const float* w3, int F, int C, int G, uint16_t* dst, hipStream_t st);
int gemm_wave_cols(int M, int N);
hipError_t launch_cast_t(const float* src, int rows, int cols, uint16_t* dst, long long ldd, hipStream_t st);

// timing.cpp: optional per-phase HIP-event timing (see bsa_timing_enable in bsa.h)
bool timing_on();
void timing_set(bool on);
void timing_select(const char* phases);
int timing_begin(const char* name, hipStream_t st);
void timing_end(int id, hipStream_t st);
hipError_t timing_query(const char* name, double* total_ms, int* count);

// Run `stmt` (kernel launches on stream st) as the timed phase `name`.
#define BSA_PHASE(name, st, stmt)                     \
  do {                                                \
    const int _tid = ::bsa::timing_begin((name), (st)); \
    stmt;                                             \
    ::bsa::timing_end(_tid, (st));                    \
  } while (0)

#define BSA_DISPATCH(FN, ...)                                                              \
  (D.bf16 ? (D.d == 64 ? FN<bf16_t, 64>(__VA_ARGS__) : FN<bf16_t, 32>(__VA_ARGS__))       \
          : (D.d == 64 ? FN<float, 64>(__VA_ARGS__) : FN<float, 32>(__VA_ARGS__)))

}  // namespace bsa
