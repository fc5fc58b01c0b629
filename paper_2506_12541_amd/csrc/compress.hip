// Block compression phi of Eq. 5: every length-l block of keys (or values) of one head,
// flattened token-major into an l*d vector with padding rows zero, maps to one coarse
// token  y = GELU_erf(x W1 + b1) W2 + b2  (or to the block mean for mean pooling).
//
// The first layer is the only sizeable contraction (l*d -> d) and runs on matrix cores
// in the storage type (bf16 MFMA with f32 accumulation for bf16 layers); x streams from
// HBM once, which bounds this kernel. The second layer (d x d) and the GELU stay in f32
// so that the compressed keys feed the top-k scoring at f32 accuracy.
#include "common.hpp"
#include "kernels.hpp"

namespace bsa {
namespace {

constexpr int kWaves = 4;
constexpr int kRB = 2;  // 16-row blocks per wave

__global__ void block_valid_kernel(const uint8_t* valid, int total_blocks, int l, uint8_t* cvalid) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total_blocks) return;
  uint8_t any = 0;
  if (valid == nullptr) {
    any = 1;
  } else {
    for (int t = 0; t < l; ++t) any |= valid[(size_t)i * l + t];
  }
  cvalid[i] = any ? 1 : 0;
}

// W1 [l*d, d] f32 -> W1^T [d, l*d] in the storage type.
template <typename T>
__global__ void transpose_w1_kernel(const float* w1, int ld, int d, T* w1t) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= ld * d) return;
  int o = i / ld, r = i % ld;
  w1t[i] = from_f32<T>(w1[(size_t)r * d + o]);
}

__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f)); }

// One wave: kRB blocks of 16 rows (coarse tokens); the workgroup stages W2 and b1/b2.
template <typename T, int HD>
__global__ void __launch_bounds__(kWaves * 64) mlp_fwd_kernel(const T* x, const uint8_t* valid, int H, int N, int l,
                                                              long long rows, const T* w1t, const float* b1,
                                                              const float* w2, const float* b2, float* out,
                                                              float* pre_out, T* out_lp) {
  constexpr int OB = HD / 16;  // 16-wide output blocks
  __shared__ float w2s[HD * HD];
  __shared__ float b1s[HD], b2s[HD];
  for (int i = threadIdx.x; i < HD * HD; i += blockDim.x) w2s[i] = w2[i];
  for (int i = threadIdx.x; i < HD; i += blockDim.x) { b1s[i] = b1[i]; b2s[i] = b2[i]; }
  __syncthreads();

  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15, j = lane >> 4;
  const int ld = l * HD;
  const int nblk = N / l;
  const long long row0 = ((long long)blockIdx.x * kWaves + wid) * (16 * kRB);

  f32x4 acc[kRB][OB];
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
    for (int ob = 0; ob < OB; ++ob) acc[rb][ob] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Per row: its flattened block and the validity of its l tokens.
  const T* xrow[kRB];
  const uint8_t* vrow[kRB];
#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
    long long row = row0 + rb * 16 + r;
    xrow[rb] = nullptr;
    vrow[rb] = nullptr;
    if (row < rows) {
      xrow[rb] = x + row * ld;
      long long bh = row / nblk;
      int blk = (int)(row % nblk);
      int b = (int)(bh / H);
      if (valid) vrow[rb] = valid + (size_t)b * N + (size_t)blk * l;
    }
  }
  // Layer 1: pre^T[o][row] = sum_i W1^T[o][i] x[row][i]; A = W1^T, B = x^T.
  for (int c = 0; c < ld / 32; ++c) {
    const int i0 = 32 * c + 8 * j;
    const int tok = i0 / HD;
    typename Chunk<T>::type bx[kRB];
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) {
      bx[rb] = zero_chunk(bx[rb]);
      if (xrow[rb] && (vrow[rb] == nullptr || vrow[rb][tok])) bx[rb] = load_chunk(xrow[rb] + i0);
    }
#pragma unroll
    for (int ob = 0; ob < OB; ++ob) {
      auto aw = load_chunk(w1t + (size_t)(16 * ob + r) * ld + i0);
#pragma unroll
      for (int rb = 0; rb < kRB; ++rb) acc[rb][ob] = mma(aw, bx[rb], acc[rb][ob]);
    }
  }

#pragma unroll
  for (int rb = 0; rb < kRB; ++rb) {
    const long long row = row0 + rb * 16 + r;   // this lane's column = row
    // hidden h[row][16 ob + 4 j + i]
    float h[OB][4];
#pragma unroll
    for (int ob = 0; ob < OB; ++ob)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        int o = 16 * ob + 4 * j + i;
        float p = acc[rb][ob][i] + b1s[o];
        acc[rb][ob][i] = p;
        h[ob][i] = gelu_erf(p);
      }
    // Layer 2 in f32 MFMA: out^T[o2][row] = sum_o W2[o][o2] h[row][o]; value e=(ob,i) of
    // lane group j is hidden unit o = 16 ob + 4 j + i.
    f32x4 y[OB];
#pragma unroll
    for (int o2b = 0; o2b < OB; ++o2b) {
      f32x4 a2 = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ob = 0; ob < OB; ++ob)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float wa = w2s[(16 * ob + 4 * j + i) * HD + 16 * o2b + r];
          a2 = __builtin_amdgcn_mfma_f32_16x16x4f32(wa, h[ob][i], a2, 0, 0, 0);
        }
      y[o2b] = a2;
    }
    if (row < rows) {
#pragma unroll
      for (int ob = 0; ob < OB; ++ob) {
        const int o = 16 * ob + 4 * j;
        float4 pv = make_float4(acc[rb][ob][0], acc[rb][ob][1], acc[rb][ob][2], acc[rb][ob][3]);
        *reinterpret_cast<float4*>(pre_out + row * HD + o) = pv;
        float4 yv = make_float4(y[ob][0] + b2s[o], y[ob][1] + b2s[o + 1], y[ob][2] + b2s[o + 2], y[ob][3] + b2s[o + 3]);
        *reinterpret_cast<float4*>(out + row * HD + o) = yv;
        out_lp[row * HD + o + 0] = from_f32<T>(yv.x);
        out_lp[row * HD + o + 1] = from_f32<T>(yv.y);
        out_lp[row * HD + o + 2] = from_f32<T>(yv.z);
        out_lp[row * HD + o + 3] = from_f32<T>(yv.w);
      }
    }
  }
}

// Mean pooling: y = (1/l) * sum of the block's real rows.
template <typename T>
__global__ void mean_pool_kernel(const T* x, const uint8_t* valid, int H, int N, int l, int hd, long long rows,
                                 float* out, T* out_lp) {
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * hd) return;
  long long row = i / hd;
  int c = (int)(i % hd);
  int nblk = N / l;
  long long bh = row / nblk;
  int blk = (int)(row % nblk);
  int b = (int)(bh / H);
  float s = 0.f;
  for (int t = 0; t < l; ++t) {
    bool ok = valid == nullptr || valid[(size_t)b * N + (size_t)blk * l + t];
    if (ok) s += to_f32<T>(x[(row * l + t) * hd + c]);
  }
  s /= (float)l;
  out[i] = s;
  out_lp[i] = from_f32<T>(s);
}

template <typename T, int HD>
hipError_t compress_impl(const Dims& D, const void* x, const uint8_t* valid, const Mlp& phi, float* out,
                         float* pre, void* out_lp, void* w1t_ws, hipStream_t st) {
  const long long rows = D.cmp_rows();
  if (D.pool == 1) {
    const long long tot = rows * HD;
    hipLaunchKernelGGL(mean_pool_kernel<T>, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, st, (const T*)x, valid,
                       D.H, D.N, D.l, HD, rows, out, (T*)out_lp);
    return hipGetLastError();
  }
  const int ld = D.l * HD;
  T* w1t = (T*)w1t_ws;
  hipLaunchKernelGGL(transpose_w1_kernel<T>, dim3((ld * HD + 255) / 256), dim3(256), 0, st, phi.w1, ld, HD, w1t);
  const long long per_wg = (long long)kWaves * 16 * kRB;
  const unsigned grid = (unsigned)((rows + per_wg - 1) / per_wg);
  hipLaunchKernelGGL((mlp_fwd_kernel<T, HD>), dim3(grid), dim3(kWaves * 64), 0, st, (const T*)x, valid, D.H, D.N,
                     D.l, rows, (const T*)w1t, phi.b1, phi.w2, phi.b2, out, pre, (T*)out_lp);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_block_valid(const Dims& D, const uint8_t* valid, uint8_t* cvalid, hipStream_t st) {
  const int total = D.B * (D.N / D.l);
  hipLaunchKernelGGL(block_valid_kernel, dim3((total + 255) / 256), dim3(256), 0, st, valid, total, D.l, cvalid);
  return hipGetLastError();
}

hipError_t launch_compress_fwd(const Dims& D, const void* x, const uint8_t* valid, const Mlp& phi, float* out,
                               float* pre, void* out_lp, void* w1t_ws, hipStream_t st) {
  if (D.bf16) {
    return D.d == 64 ? compress_impl<bf16_t, 64>(D, x, valid, phi, out, pre, out_lp, w1t_ws, st)
                     : compress_impl<bf16_t, 32>(D, x, valid, phi, out, pre, out_lp, w1t_ws, st);
  }
  return D.d == 64 ? compress_impl<float, 64>(D, x, valid, phi, out, pre, out_lp, w1t_ws, st)
                   : compress_impl<float, 32>(D, x, valid, phi, out, pre, out_lp, w1t_ws, st);
}

}  // namespace bsa
