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
  float scale;         // softmax scale
  long long rows() const { return (long long)B * H * N; }
  long long cmp_rows() const { return (long long)B * H * (N / l); }
};

struct Mlp { const float *w1, *b1, *w2, *b2; };
struct MlpGrad { float *w1, *b1, *w2, *b2; };

// tree.hip
size_t tree_workspace_bytes(int64_t n_real, int64_t n_pad, int batch);
hipError_t launch_build_tree(const float* pts, int64_t n_real, int dim, int64_t n_pad, int batch,
                             int* perm, void* ws, hipStream_t st);
hipError_t launch_permute(const void* src, const int* perm, int64_t n_real, int64_t n_pad, int batch,
                          int heads, int hd, int dtype, void* dst, uint8_t* valid, bool inverse,
                          hipStream_t st);

// compress.hip: compression phi of Eq. 5 and its backward
hipError_t launch_block_valid(const Dims& D, const uint8_t* valid, uint8_t* cvalid, hipStream_t st);
hipError_t launch_compress_fwd(const Dims& D, const void* x, const uint8_t* valid, const Mlp& phi,
                               float* out, float* pre, void* out_lp, void* w1t_ws, hipStream_t st);

// select.hip: pooled-query block scores and group top-k (Eq. 6, 7, 10-12)
hipError_t launch_select_topk(const Dims& D, const void* q, const uint8_t* valid, const float* kcmp,
                              const uint8_t* cvalid, int* sel, hipStream_t st);

// attn_fwd.hip: the three attention branches (Eq. 3, 5, 8) and the gate (Eq. 9)
hipError_t launch_ball_fwd(const Dims& D, const void* q, const void* k, const void* v, const uint8_t* valid,
                           void* o, float* lse, hipStream_t st);
hipError_t launch_cmp_fwd(const Dims& D, const void* q, const void* kc, const void* vc, const uint8_t* valid,
                          const uint8_t* cvalid, void* o, float* lse, hipStream_t st);
hipError_t launch_slc_fwd(const Dims& D, const void* q, const void* k, const void* v, const uint8_t* valid,
                          const int* sel, void* o, float* lse, hipStream_t st);
hipError_t launch_gate_fwd(const Dims& D, const void* ob, const float* gate, const uint8_t* valid, void* o,
                           hipStream_t st);

}  // namespace bsa
