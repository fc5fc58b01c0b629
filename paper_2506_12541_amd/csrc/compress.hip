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
#include "attn_common.hpp"

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

// One compression of a forward launch: its input rows, weights (W1 transposed, in the storage
// type) and outputs.
struct MlpFwdJob {
  const void* x;
  const void* w1t;
  const float *b1, *w2, *b2;
  float *out, *pre;
  void* out_lp;
  float lp_scale;
};

// One wave: kRB blocks of 16 rows (coarse tokens); the workgroup stages W2 and b1/b2.
// grid.y picks the job (the key and value compressions share one launch).
template <typename T, int HD>
__global__ void __launch_bounds__(kWaves * 64) mlp_fwd_kernel(const uint8_t* valid, int H, int N, int l,
                                                              long long rows, MlpFwdJob j0, MlpFwdJob j1) {
  const MlpFwdJob& job = blockIdx.y ? j1 : j0;
  const T* x = (const T*)job.x;
  const T* w1t = (const T*)job.w1t;
  const float *b1 = job.b1, *w2 = job.w2, *b2 = job.b2;
  float *out = job.out, *pre_out = job.pre;
  T* out_lp = (T*)job.out_lp;
  const float lp_scale = job.lp_scale;
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
  // Layer 1: pre^T[o][row] = sum_i W1^T[o][i] x[row][i]; A = W1^T, B = x^T. The operands of
  // chunk c + 1 are loaded while chunk c is multiplied.
  typedef typename Chunk<T>::type CT;
  CT bx[2][kRB], aw[2][OB];
  auto fetch = [&](int c, CT (&bxs)[kRB], CT (&aws)[OB]) {
    const int i0 = 32 * c + 8 * j;
    const int tok = i0 / HD;
#pragma unroll
    for (int rb = 0; rb < kRB; ++rb) {
      bxs[rb] = zero_chunk(bxs[rb]);
      if (xrow[rb] && (vrow[rb] == nullptr || vrow[rb][tok])) bxs[rb] = load_chunk(xrow[rb] + i0);
    }
#pragma unroll
    for (int ob = 0; ob < OB; ++ob) aws[ob] = load_chunk(w1t + (size_t)(16 * ob + r) * ld + i0);
  };
  auto mult = [&](const CT (&bxs)[kRB], const CT (&aws)[OB]) {
#pragma unroll
    for (int ob = 0; ob < OB; ++ob)
#pragma unroll
      for (int rb = 0; rb < kRB; ++rb) acc[rb][ob] = mma(aws[ob], bxs[rb], acc[rb][ob]);
  };
  const int nc = ld / 32;   // even: l*d is a multiple of 64
  fetch(0, bx[0], aw[0]);
  for (int c = 0; c < nc; c += 2) {
    fetch(c + 1, bx[1], aw[1]);
    mult(bx[0], aw[0]);
    if (c + 2 < nc) fetch(c + 2, bx[0], aw[0]);
    mult(bx[1], aw[1]);
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
        out_lp[row * HD + o + 0] = from_f32<T>(yv.x * lp_scale);
        out_lp[row * HD + o + 1] = from_f32<T>(yv.y * lp_scale);
        out_lp[row * HD + o + 2] = from_f32<T>(yv.z * lp_scale);
        out_lp[row * HD + o + 3] = from_f32<T>(yv.w * lp_scale);
      }
    }
  }
}

// Mean pooling: y = (1/l) * sum of the block's real rows.
template <typename T>
__global__ void mean_pool_kernel(const T* x, const uint8_t* valid, int H, int N, int l, int hd, long long rows,
                                 float* out, T* out_lp, float lp_scale) {
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
  out_lp[i] = from_f32<T>(s * lp_scale);
}

// ---------------------------------------------------------------------------------
// Backward of phi. With y = h W2 + b2, h = GELU(pre), pre = x W1 + b1 (per row = block):
//   dh = dy W2^T, dpre = dh * GELU'(pre), dx = dpre W1^T,
//   dW2 = h^T dy, db2 = sum dy, dW1 = x^T dpre, db1 = sum dpre   (sums over all rows).
// Rows are split into fixed chunks whose weight-gradient partials are summed in order.
// ---------------------------------------------------------------------------------
__device__ __forceinline__ float gelu_erf_grad(float x) {
  return 0.5f * (1.0f + erff(x * 0.70710678118654752f)) + x * 0.3989422804014327f * __expf(-0.5f * x * x);
}

// One wave per 16 rows: dpre (stored), and dx = dpre W1^T added into the token gradients.
// The dx product runs in the storage type (bf16 MFMA for bf16 layers; W1 holds
// bf16-representable values there), the rest in f32.
template <typename T, int HD>
__global__ void __launch_bounds__(256) mlp_bwd_rows_kernel(const float* dy, const float* pre, const uint8_t* valid,
                                                           int H, int N, int l, long long rows, const T* w1,
                                                           const float* w2, float* dpre_out, float* dx_accum) {
  constexpr int NCH = HD / 32, OB = HD / 16;
  __shared__ float w2s[HD * (HD + 4)];
  __shared__ __attribute__((aligned(16))) float dps_all[4][16 * (HD + 4)];
  for (int i = threadIdx.x; i < HD * HD; i += blockDim.x) w2s[(i / HD) * (HD + 4) + i % HD] = w2[i];
  __syncthreads();
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15, j = lane >> 4;
  const long long row0 = ((long long)blockIdx.x * 4 + wid) * 16;
  const long long row = row0 + r;
  const bool rok = row < rows;
  float* dps = dps_all[wid];
  // dh^T[o][row] = sum_o2 W2[o][o2] dy[row][o2]; A = W2 rows (o), B = dy^T
  f32x8 by[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) by[c] = rok ? load_chunk(dy + row * HD + 32 * c + 8 * j) : f32x8{};
#pragma unroll
  for (int ob = 0; ob < OB; ++ob) {
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      f32x8 a;
#pragma unroll
      for (int e = 0; e < 8; ++e) a[e] = w2s[(16 * ob + r) * (HD + 4) + 32 * c + 8 * j + e];
      acc = mma(a, by[c], acc);
    }
    // lane: row r, hidden units o = 16 ob + 4 j + i
    float4 pv = rok ? *reinterpret_cast<const float4*>(pre + row * HD + 16 * ob + 4 * j) : make_float4(0, 0, 0, 0);
    const float pa[4] = {pv.x, pv.y, pv.z, pv.w};
    float d4[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) d4[i] = acc[i] * gelu_erf_grad(pa[i]);
    *reinterpret_cast<float4*>(&dps[r * (HD + 4) + 16 * ob + 4 * j]) = make_float4(d4[0], d4[1], d4[2], d4[3]);
    if (rok) *reinterpret_cast<float4*>(dpre_out + row * HD + 16 * ob + 4 * j) = make_float4(d4[0], d4[1], d4[2], d4[3]);
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  // dx^T[i][row] = sum_o W1[i][o] dpre[row][o]; A = W1 rows (i), B = dpre^T
  typename Chunk<T>::type bd[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) bd[c] = make_chunk<T>(&dps[r * (HD + 4) + 32 * c + 8 * j]);
  const int ld = l * HD;
  const int nblk = N / l;
  long long bhh = rok ? row / nblk : 0;
  const int blk = rok ? (int)(row % nblk) : 0;
  const int b = (int)(bhh / H);
  for (int ib = 0; ib < ld / 16; ++ib) {
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NCH; ++c) acc = mma(load_chunk(w1 + (size_t)(16 * ib + r) * HD + 32 * c + 8 * j), bd[c], acc);
    // lane: row r, flat indices i = 16 ib + 4 j + t (one token, 4 consecutive channels)
    const int i0 = 16 * ib + 4 * j;
    const int tok = i0 / HD, ch = i0 % HD;
    if (rok && (valid == nullptr || valid[(size_t)b * N + (size_t)blk * l + tok])) {
      float* dst = dx_accum + (row * l + tok) * HD + ch;
      float4 o = *reinterpret_cast<float4*>(dst);
      o.x += acc[0]; o.y += acc[1]; o.z += acc[2]; o.w += acc[3];
      *reinterpret_cast<float4*>(dst) = o;
    }
  }
}

template <typename T>
__global__ void cast_w_kernel(const float* x, int n, T* y) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) y[i] = from_f32<T>(x[i]);
}

// dW1 partials: workgroup = (64 flattened inputs i, row chunk); wave w owns i in [16w, 16w+16).
template <typename T, int HD>
__global__ void __launch_bounds__(256) mlp_bwd_w1_kernel(const T* x, const uint8_t* valid, const float* dpre, int H,
                                                         int N, int l, long long rows, long long rows_per_chunk,
                                                         float* part) {
  constexpr int TSTR = 32 + 4;
  constexpr int OB = HD / 16;
  typedef typename Chunk<T>::type CT;
  __shared__ __attribute__((aligned(16))) T xt[64 * TSTR];
  __shared__ __attribute__((aligned(16))) T dt[HD * TSTR];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15, j = lane >> 4;
  const int ld = l * HD;
  const int i0 = blockIdx.x * 64;
  const int chunk = blockIdx.y;
  const long long rbeg = chunk * rows_per_chunk;
  const long long rend = rbeg + rows_per_chunk < rows ? rbeg + rows_per_chunk : rows;
  const int nblk = N / l;
  f32x4 acc[OB];
#pragma unroll
  for (int ob = 0; ob < OB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (long long r0 = rbeg; r0 < rend; r0 += 32) {
    __syncthreads();
    // x^T tile [64 i][32 rows]: items of 4 rows x 8 columns
    for (int e = threadIdx.x; e < 8 * 8; e += 256) {
      const int kq = e / 8, dc = (e % 8) * 8;
      const int tok = (i0 + dc) / HD;
      const T* rp[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const long long row = r0 + 4 * kq + u;
        bool ok = row < rend;
        if (ok && valid) {
          const long long bhh = row / nblk;
          const int blk = (int)(row % nblk);
          ok = valid[(size_t)(bhh / H) * N + (size_t)blk * l + tok] != 0;
        }
        rp[u] = ok ? x + row * ld + i0 : nullptr;
      }
      stage_t(rp, dc, xt, TSTR, 4 * kq);
    }
    // dpre^T tile [HD][32 rows]
    for (int e = threadIdx.x; e < 8 * (HD / 8); e += 256) {
      const int kq = e / (HD / 8), dc = (e % (HD / 8)) * 8;
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) {
        float v4[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const long long row = r0 + 4 * kq + u;
          v4[u] = row < rend ? dpre[row * HD + dc + cc] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) dt[(dc + cc) * TSTR + 4 * kq + u] = from_f32<T>(v4[u]);
      }
    }
    __syncthreads();
    // D[i][o] += sum_rows xt[i][row] dt[o][row]; contraction over 32 rows = one chunk
    CT a = load_4x2(&xt[(16 * wid + r) * TSTR + 4 * j]);
#pragma unroll
    for (int ob = 0; ob < OB; ++ob) acc[ob] = mma(a, load_4x2(&dt[(16 * ob + r) * TSTR + 4 * j]), acc[ob]);
  }
  // lane: o = 16 ob + r (column), i = i0 + 16 wid + 4 j + t (rows)
  float* out = part + (size_t)chunk * ld * HD;
#pragma unroll
  for (int ob = 0; ob < OB; ++ob)
#pragma unroll
    for (int t = 0; t < 4; ++t) out[(size_t)(i0 + 16 * wid + 4 * j + t) * HD + 16 * ob + r] = acc[ob][t];
}

// dW2, db1, db2 partials over a row chunk: thread (o2, o-slice).
template <int HD>
__global__ void __launch_bounds__(256) mlp_bwd_small_kernel(const float* dy, const float* pre, const float* dpre,
                                                            long long rows, long long rows_per_chunk, float* part) {
  __shared__ float hs[32][HD];
  __shared__ float ys[32][HD];
  __shared__ float ps[32][HD];
  const int chunk = blockIdx.x;
  const long long rbeg = chunk * rows_per_chunk;
  const long long rend = rbeg + rows_per_chunk < rows ? rbeg + rows_per_chunk : rows;
  constexpr int PER = HD * HD / 256;  // dW2 entries per thread
  const int o2 = threadIdx.x % HD;
  const int ob = (threadIdx.x / HD) * PER;
  float acc[PER];
#pragma unroll
  for (int t = 0; t < PER; ++t) acc[t] = 0.f;
  float sb1 = 0.f, sb2 = 0.f;
  for (long long r0 = rbeg; r0 < rend; r0 += 32) {
    __syncthreads();
    for (int e = threadIdx.x; e < 32 * HD; e += 256) {
      const int rr = e / HD, c = e % HD;
      const long long row = r0 + rr;
      float pv = 0.f, yv = 0.f, dv = 0.f;
      if (row < rend) {
        pv = pre[row * HD + c];
        yv = dy[row * HD + c];
        dv = dpre[row * HD + c];
      }
      hs[rr][c] = row < rend ? gelu_erf(pv) : 0.f;
      ys[rr][c] = yv;
      ps[rr][c] = dv;
    }
    __syncthreads();
    for (int rr = 0; rr < 32; ++rr) {
      const float y = ys[rr][o2];
#pragma unroll
      for (int t = 0; t < PER; ++t) acc[t] += hs[rr][ob + t] * y;
      if (threadIdx.x < HD) { sb1 += ps[rr][o2]; sb2 += y; }
    }
  }
  float* out = part + (size_t)chunk * (HD * HD + 2 * HD);
#pragma unroll
  for (int t = 0; t < PER; ++t) out[(ob + t) * HD + o2] = acc[t];
  if (threadIdx.x < HD) {
    out[HD * HD + o2] = sb1;
    out[HD * HD + HD + o2] = sb2;
  }
}

// out[i] = sum over chunks of part[c * stride + i]. A workgroup owns 64 outputs; its
// 4 waves each sum every 4th chunk, then the four partial sums are added in wave order.
__global__ void __launch_bounds__(256) sum_parts_kernel(const float* part, int chunks, long long n, long long stride,
                                                        float* out) {
  __shared__ float red[4][64];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const long long i = (long long)blockIdx.x * 64 + lane;
  float s = 0.f;
  if (i < n)
    for (int c = wid; c < chunks; c += 4) s += part[(long long)c * stride + i];
  red[wid][lane] = s;
  __syncthreads();
  if (wid == 0 && i < n) out[i] = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
}

// Mean pooling backward: every real token of a block receives dy / l.
__global__ void mean_pool_bwd_kernel(const float* dy, const uint8_t* valid, int H, int N, int l, int hd, long long rows,
                                     float* dx_accum) {
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * l * hd) return;
  const int c = (int)(i % hd);
  const long long tokrow = i / hd;          // (b*H + h) * N + n
  const long long row = tokrow / l;         // block row
  const int t = (int)(tokrow % l);
  const int nblk = N / l;
  const long long bhh = row / nblk;
  const int blk = (int)(row % nblk);
  const int b = (int)(bhh / H);
  if (valid && !valid[(size_t)b * N + (size_t)blk * l + t]) return;
  dx_accum[i] += dy[row * hd + c] / (float)l;
}

// ---- bf16 layers: the backward of phi in four passes (both layers' weight gradients as
// deterministic chunk partials, summed in order) ----

// (1) Per 32-row tile, on the vector ALU in f32: dh = dy W2^T, dpre = dh GELU'(pre) (stored
// in f32 and bf16), and this workgroup's partials of dW2 = h^T dy, db1 = sum dpre,
// db2 = sum dy over its rows. Register blocking keeps LDS traffic low: for dh a thread
// owns 2 rows x 4 outputs (W2 staged transposed so its 4 outputs are one float4 read), for
// dW2 a 4 x 4 block.
template <int HD>
__global__ void __launch_bounds__(256) mlp_bwd_pre_kernel(const float* dy, const float* pre, const float* w2,
                                                          long long rows, long long rows_per_wg, float* dpre,
                                                          bf16_t* dpre_lp, float* part) {
  constexpr int TR = 32;                       // rows per tile
  constexpr int OQ = HD / 4;                   // 4-wide output groups per row
  constexpr int RB = TR * OQ / 256;            // rows per thread in the dh pass (2 for HD=64, 1 for 32)
  constexpr int NB4 = (HD / 4) * (HD / 4);      // 4x4 dW2 blocks (at most one per thread)
  constexpr int W2B = 1;
  static_assert(NB4 <= 256, "dW2 blocks");
  static_assert(RB >= 1 && TR * OQ % 256 == 0, "tile split");
  __shared__ __attribute__((aligned(16))) float w2t[HD][HD + 4];   // W2^T: w2t[o2][o] = W2[o][o2]
  __shared__ __attribute__((aligned(16))) float hs[TR][HD + 4], ys[TR][HD + 4], ps[TR][HD + 4];
  for (int i = threadIdx.x; i < HD * HD; i += 256) w2t[i % HD][i / HD] = w2[i];
  const long long rbeg = blockIdx.x * rows_per_wg;
  const long long rend = rbeg + rows_per_wg < rows ? rbeg + rows_per_wg : rows;
  const int t = threadIdx.x;
  const int oq = t % OQ;             // dh pass: outputs 4 oq .. 4 oq + 3
  const int rr0 = (t / OQ) * RB;     // dh pass: rows rr0 .. rr0 + RB - 1
  f32x4 aw2[W2B][4];                 // dW2 pass: block (o rows 4 bo + u, o2 4 bq .. + 3)
#pragma unroll
  for (int w = 0; w < W2B; ++w)
#pragma unroll
    for (int u = 0; u < 4; ++u) aw2[w][u] = f32x4{0.f, 0.f, 0.f, 0.f};
  float ab1 = 0.f, ab2 = 0.f;
  for (long long r0 = rbeg; r0 < rend; r0 += TR) {
    __syncthreads();
    for (int e = t; e < TR * OQ; e += 256) {
      const int rr = e / OQ, c = 4 * (e % OQ);
      const long long row = r0 + rr;
      float4 pv = make_float4(0.f, 0.f, 0.f, 0.f), yv = pv;
      if (row < rend) {
        pv = *reinterpret_cast<const float4*>(pre + row * HD + c);
        yv = *reinterpret_cast<const float4*>(dy + row * HD + c);
      }
      *reinterpret_cast<float4*>(&ys[rr][c]) = yv;
      *reinterpret_cast<float4*>(&hs[rr][c]) = make_float4(gelu_erf(pv.x), gelu_erf(pv.y), gelu_erf(pv.z), gelu_erf(pv.w));
      *reinterpret_cast<float4*>(&ps[rr][c]) = pv;   // pre, replaced by dpre below
    }
    __syncthreads();
    f32x4 dh[RB];
#pragma unroll
    for (int u = 0; u < RB; ++u) dh[u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
    for (int o2 = 0; o2 < HD; ++o2) {
      const float4 wv = *reinterpret_cast<const float4*>(&w2t[o2][4 * oq]);
#pragma unroll
      for (int u = 0; u < RB; ++u) {
        const float yv = ys[rr0 + u][o2];
        dh[u][0] += yv * wv.x; dh[u][1] += yv * wv.y; dh[u][2] += yv * wv.z; dh[u][3] += yv * wv.w;
      }
    }
    float4 dv[RB];
#pragma unroll
    for (int u = 0; u < RB; ++u) {
      const int rr = rr0 + u;
      const long long row = r0 + rr;
      const float4 pv = *reinterpret_cast<const float4*>(&ps[rr][4 * oq]);
      const bool ok = row < rend;
      dv[u] = ok ? make_float4(dh[u][0] * gelu_erf_grad(pv.x), dh[u][1] * gelu_erf_grad(pv.y),
                               dh[u][2] * gelu_erf_grad(pv.z), dh[u][3] * gelu_erf_grad(pv.w))
                 : make_float4(0.f, 0.f, 0.f, 0.f);
      if (ok) {
        *reinterpret_cast<float4*>(dpre + row * HD + 4 * oq) = dv[u];
        const uint32_t lo = (uint32_t)f2bf(dv[u].x) | ((uint32_t)f2bf(dv[u].y) << 16);
        const uint32_t hi = (uint32_t)f2bf(dv[u].z) | ((uint32_t)f2bf(dv[u].w) << 16);
        *reinterpret_cast<uint2*>(dpre_lp + row * HD + 4 * oq) = make_uint2(lo, hi);
      }
    }
    __syncthreads();   // every thread has read its pre values
#pragma unroll
    for (int u = 0; u < RB; ++u) *reinterpret_cast<float4*>(&ps[rr0 + u][4 * oq]) = dv[u];
    __syncthreads();
    // dW2 blocks: thread owns o = 4 bo + u, o2 = 4 bq .. + 3
#pragma unroll
    for (int w = 0; w < W2B; ++w) {
      const int blk = t * W2B + w;
      const int bo = blk / OQ, bq = blk % OQ;
      if (blk >= NB4) continue;
#pragma unroll 4
      for (int rr = 0; rr < TR; ++rr) {
        const float4 hv = *reinterpret_cast<const float4*>(&hs[rr][4 * bo]);
        const float4 yv = *reinterpret_cast<const float4*>(&ys[rr][4 * bq]);
        const float h4[4] = {hv.x, hv.y, hv.z, hv.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          aw2[w][u][0] += h4[u] * yv.x; aw2[w][u][1] += h4[u] * yv.y;
          aw2[w][u][2] += h4[u] * yv.z; aw2[w][u][3] += h4[u] * yv.w;
        }
      }
    }
    if (t < HD) {
#pragma unroll 8
      for (int rr = 0; rr < TR; ++rr) { ab1 += ps[rr][t]; ab2 += ys[rr][t]; }
    }
  }
  float* out = part + (size_t)blockIdx.x * (HD * HD + 2 * HD);
  {
#pragma unroll
    for (int w = 0; w < W2B; ++w) {
      const int blk = t * W2B + w;
      const int bo = blk / OQ, bq = blk % OQ;
      if (blk >= NB4) continue;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        *reinterpret_cast<float4*>(out + (4 * bo + u) * HD + 4 * bq) =
            make_float4(aw2[w][u][0], aw2[w][u][1], aw2[w][u][2], aw2[w][u][3]);
    }
  }
  if (t < HD) {
    out[HD * HD + t] = ab1;
    out[HD * HD + HD + t] = ab2;
  }
}

// (2) dx = dpre W1^T added into the token gradients, as C^T = W1 dpre^T on bf16 matrix
// cores: a workgroup owns 256 flattened inputs i (their W1 rows staged in LDS by direct
// loads) and 64 block rows per pass (wave w: rows 16w..16w+15, its dpre fragments from
// global); a lane ends with 4 consecutive i of one row per 16-input tile. All tiles of a
// pass are computed first, then the gradient rows are read together and written back.
template <int HD>
__global__ void __launch_bounds__(256) mlp_bwd_dx_kernel(const bf16_t* dpre_lp, const bf16_t* w1, const uint8_t* valid,
                                                         int H, int N, int l, long long rows, int passes,
                                                         float* dx_accum) {
  constexpr int NCH = HD / 32;
  constexpr int IT = 256 / 16;   // i tiles per workgroup
  __shared__ __attribute__((aligned(16))) bf16_t w1s[256 * HD];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15, j = lane >> 4;
  const int ld = l * HD;
  const int i0 = blockIdx.x * 256;
  dma_tile<HD, 256, 4>(w1s, w1, i0, ld, wid, lane);
  vm_drain();
  __syncthreads();
  const int nblk = N / l;
  for (int pz = 0; pz < passes; ++pz) {
    const long long row0 = ((long long)blockIdx.y * passes + pz) * 64 + 16 * wid;
    if (row0 >= rows) break;
    const long long row = row0 + r;
    const bool rok = row < rows;
    bf16x8 bd[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c)
      bd[c] = rok ? load_chunk(dpre_lp + row * HD + 32 * c + 8 * j) : zero_chunk(bd[c]);
    const long long bhh = rok ? row / nblk : 0;
    const int blk = rok ? (int)(row % nblk) : 0;
    const int b = (int)(bhh / H);
    f32x4 acc[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      acc[it] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NCH; ++c) acc[it] = mma(lds_row_chunk<HD>(w1s, 16 * it + r, 4 * c + j), bd[c], acc[it]);
    }
    // lane: row r, flat inputs i = i0 + 16 it + 4 j + t (one token, 4 consecutive channels)
    float4 old[IT];
    bool ok[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int i = i0 + 16 * it + 4 * j;
      const int tok = i / HD, ch = i % HD;
      ok[it] = rok && (valid == nullptr || valid[(size_t)b * N + (size_t)blk * l + tok]);
      old[it] = ok[it] ? *reinterpret_cast<const float4*>(dx_accum + (row * l + tok) * HD + ch)
                       : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
      const int i = i0 + 16 * it + 4 * j;
      const int tok = i / HD, ch = i % HD;
      if (ok[it])
        *reinterpret_cast<float4*>(dx_accum + (row * l + tok) * HD + ch) =
            make_float4(old[it].x + acc[it][0], old[it].y + acc[it][1], old[it].z + acc[it][2], old[it].w + acc[it][3]);
    }
  }
}

// (3) dW1 partials over a chunk of block rows, D[i][o] = sum_rows x[row][i] dpre[row][o],
// on bf16 matrix cores: a workgroup owns 256 flattened inputs i (wave w: 64 of them) and
// walks its rows 32 at a time; the x and dpre tiles are double-buffered in LDS (two
// distinct objects, loop unrolled by two) by direct loads, and both operands, which run
// along the rows, come from transpose reads. Inputs of padding tokens are zeroed in LDS.
template <int HD>
__global__ void __launch_bounds__(256) mlp_bwd_w1_dma_kernel(const bf16_t* x, const uint8_t* valid,
                                                             const bf16_t* dpre_lp, int H, int N, int l,
                                                             long long rows, long long rows_per_chunk, float* part) {
  constexpr int XW = 256;          // inputs per workgroup (tile width)
  constexpr int OB = HD / 16;
  constexpr int TR = 32;           // rows per step
  __shared__ __attribute__((aligned(16))) bf16_t xs0[TR * XW], xs1[TR * XW];
  __shared__ __attribute__((aligned(16))) bf16_t ds0[TR * HD], ds1[TR * HD];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15;
  const int ld = l * HD;
  const int i0 = blockIdx.x * XW;
  const long long rbeg = (long long)blockIdx.y * rows_per_chunk;
  const long long rend = rbeg + rows_per_chunk < rows ? rbeg + rows_per_chunk : rows;
  const int nblk = N / l;
  const bf16_t* xb = x + i0;   // column offset of this workgroup's inputs
  auto issue = [&](long long r0, bf16_t* xd, bf16_t* dd) {
    // x rows are ld elements apart: load each row's 256-input slice as its own 512-byte run
#pragma unroll
    for (int u = 0; u < TR * XW / 8 / 64 / 4; ++u) {
      const int blkk = wid * (TR * XW / 8 / 64 / 4) + u;     // 1 KB LDS block
      const int idx = blkk * 64 + lane;                      // 16-byte chunk of the tile
      const int row = idx / (XW / 8);
      const int lc = (idx % (XW / 8)) ^ swz<XW>(row);
      const long long gr = r0 + row < rend ? r0 + row : rend - 1;
      __builtin_amdgcn_global_load_lds(xb + gr * ld + 8 * lc, xd + blkk * 512, 16, 0, 0);
    }
    constexpr int NID = TR * HD * 2 / 1024;   // 1 KB blocks of the dpre tile
    if constexpr (NID >= 4) {
      dma_tile<HD, TR, 4>(dd, dpre_lp, (int)r0, (int)rend, wid, lane);
    } else {
      if (wid < NID) dma_tile<HD, TR, NID>(dd, dpre_lp, (int)r0, (int)rend, wid, lane);
    }
  };
  f32x4 acc[4][OB];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int ob = 0; ob < OB; ++ob) acc[a][ob] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto step = [&](long long r0, bf16_t* xc, bf16_t* dc, bf16_t* xn, bf16_t* dn) {
    vm_drain();
    __syncthreads();
    const bool tail = r0 + TR > rend;
    if (valid != nullptr || tail) {   // zero inputs of padding tokens and rows past the chunk
      for (int e = threadIdx.x; e < TR * (XW / HD); e += 256) {
        const int rr = e / (XW / HD), tk = e % (XW / HD);
        const long long row = r0 + rr;
        bool ok = row < rend;
        if (ok && valid) {
          const long long bhh = row / nblk;
          const int blk = (int)(row % nblk);
          ok = valid[(size_t)(bhh / H) * N + (size_t)blk * l + (i0 + tk * HD) / HD] != 0;
        }
        if (!ok)
          for (int c = 0; c < HD / 8; ++c)
            *reinterpret_cast<uint4*>(&xc[rr * XW + 8 * (((tk * HD) / 8 + c) ^ swz<XW>(rr))]) = make_uint4(0, 0, 0, 0);
      }
      __syncthreads();
    }
    if (r0 + TR < rend) issue(r0 + TR, xn, dn);
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const bf16x8 ax = lds_tr_chunk<XW>(xc, 0, 64 * wid + 16 * a, lane);
#pragma unroll
      for (int ob = 0; ob < OB; ++ob) acc[a][ob] = mma(ax, lds_tr_chunk<HD>(dc, 0, 16 * ob, lane), acc[a][ob]);
    }
  };
  issue(rbeg, xs0, ds0);
  for (long long r0 = rbeg; r0 < rend; r0 += 2 * TR) {
    step(r0, xs0, ds0, xs1, ds1);
    if (r0 + TR < rend) step(r0 + TR, xs1, ds1, xs0, ds0);
  }
  // lane: o = 16 ob + r (column), i = i0 + 64 wid + 16 a + 4 j + t (rows)
  const int j = lane >> 4;
  float* out = part + (size_t)blockIdx.y * ld * HD;
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int ob = 0; ob < OB; ++ob)
#pragma unroll
      for (int t = 0; t < 4; ++t) out[(size_t)(i0 + 64 * wid + 16 * a + 4 * j + t) * HD + 16 * ob + r] = acc[a][ob][t];
}

// (4) out[i] = sum over chunks of part[c * stride + i], chunks in order; a workgroup owns
// 64 outputs and its 4 waves take every 4th chunk, then add their sums in wave order.
__global__ void __launch_bounds__(256) sum_parts_wide_kernel(const float* part, int chunks, long long n,
                                                             long long stride, float* out) {
  __shared__ float red[4][64];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const long long i = (long long)blockIdx.x * 64 + lane;
  float s = 0.f;
  if (i < n) {
#pragma unroll 8
    for (int c = wid; c < chunks; c += 4) s += part[(long long)c * stride + i];
  }
  red[wid][lane] = s;
  __syncthreads();
  if (wid == 0 && i < n) out[i] = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
}

template <int HD>
hipError_t compress_bwd_bf16(const Dims& D, const void* x, const uint8_t* valid, const Mlp& phi, const float* pre,
                             const float* dy, float* dx_accum, const MlpGrad& grad, const MlpBwdWs& ws,
                             hipStream_t st) {
  const long long rows = D.cmp_rows();
  const int ld = D.l * HD;
  bf16_t* w1 = (bf16_t*)ws.w1_lp;
  bf16_t* dpl = (bf16_t*)ws.dpre_lp;
  hipLaunchKernelGGL(cast_w_kernel<bf16_t>, dim3((ld * HD + 255) / 256), dim3(256), 0, st, phi.w1, ld * HD, w1);
  const long long rps = ((rows + ws.chunks_small - 1) / ws.chunks_small + 31) / 32 * 32;
  hipLaunchKernelGGL((mlp_bwd_pre_kernel<HD>), dim3(ws.chunks_small), dim3(256), 0, st, dy, pre, phi.w2, rows, rps,
                     ws.dpre, dpl, ws.part_small);
  constexpr int kPasses = 4;   // 64-row passes per workgroup of the dx product
  const long long ry = (rows + 64 * kPasses - 1) / (64 * kPasses);
  hipLaunchKernelGGL((mlp_bwd_dx_kernel<HD>), dim3(ld / 256, (unsigned)ry), dim3(256), 0, st, (const bf16_t*)dpl,
                     (const bf16_t*)w1, valid, D.H, D.N, D.l, rows, kPasses, dx_accum);
  const long long rpc = ((rows + ws.chunks - 1) / ws.chunks + 31) / 32 * 32;
  const int nch = (int)((rows + rpc - 1) / rpc);
  hipLaunchKernelGGL((mlp_bwd_w1_dma_kernel<HD>), dim3(ld / 256, nch), dim3(256), 0, st, (const bf16_t*)x, valid,
                     (const bf16_t*)dpl, D.H, D.N, D.l, rows, rpc, ws.part_w1);
  const long long n1 = (long long)ld * HD;
  hipLaunchKernelGGL(sum_parts_wide_kernel, dim3((unsigned)((n1 + 63) / 64)), dim3(256), 0, st, ws.part_w1, nch, n1,
                     n1, grad.w1);
  const long long ss = (long long)HD * HD + 2 * HD;
  const int nsm = (int)((rows + rps - 1) / rps);
  float* tmp = grad.w2;   // W2, b1, b2 partials are summed into their three outputs
  hipLaunchKernelGGL(sum_parts_wide_kernel, dim3((HD * HD + 63) / 64), dim3(256), 0, st, ws.part_small, nsm,
                     (long long)HD * HD, ss, tmp);
  hipLaunchKernelGGL(sum_parts_wide_kernel, dim3(1), dim3(256), 0, st, ws.part_small + HD * HD, nsm, (long long)HD,
                     ss, grad.b1);
  hipLaunchKernelGGL(sum_parts_wide_kernel, dim3(1), dim3(256), 0, st, ws.part_small + HD * HD + HD, nsm,
                     (long long)HD, ss, grad.b2);
  return hipGetLastError();
}

template <typename T, int HD>
hipError_t compress_bwd_impl(const Dims& D, const void* x, const uint8_t* valid, const Mlp& phi, const float* pre,
                             const float* dy, float* dx_accum, const MlpGrad& grad, const MlpBwdWs& ws,
                             hipStream_t st) {
  const long long rows = D.cmp_rows();
  if (D.pool == 1) {
    const long long tot = rows * D.l * HD;
    hipLaunchKernelGGL(mean_pool_bwd_kernel, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, st, dy, valid, D.H, D.N,
                       D.l, HD, rows, dx_accum);
    return hipGetLastError();
  }
  if constexpr (sizeof(T) == 2) {
    if (D.l * HD % 256 == 0) return compress_bwd_bf16<HD>(D, x, valid, phi, pre, dy, dx_accum, grad, ws, st);
  }
  const int ld = D.l * HD;
  const T* w1 = (const T*)phi.w1;
  if (sizeof(T) == 2) {
    hipLaunchKernelGGL(cast_w_kernel<T>, dim3((ld * HD + 255) / 256), dim3(256), 0, st, phi.w1, ld * HD, (T*)ws.w1_lp);
    w1 = (const T*)ws.w1_lp;
  }
  hipLaunchKernelGGL((mlp_bwd_rows_kernel<T, HD>), dim3((unsigned)((rows + 63) / 64)), dim3(256), 0, st, dy, pre, valid,
                     D.H, D.N, D.l, rows, w1, phi.w2, ws.dpre, dx_accum);
  const long long rpc = ((rows + ws.chunks - 1) / ws.chunks + 31) / 32 * 32;
  hipLaunchKernelGGL((mlp_bwd_w1_kernel<T, HD>), dim3(ld / 64, ws.chunks), dim3(256), 0, st, (const T*)x, valid, ws.dpre,
                     D.H, D.N, D.l, rows, rpc, ws.part_w1);
  const long long rps = ((rows + ws.chunks_small - 1) / ws.chunks_small + 31) / 32 * 32;
  hipLaunchKernelGGL((mlp_bwd_small_kernel<HD>), dim3(ws.chunks_small), dim3(256), 0, st, dy, pre, ws.dpre, rows, rps,
                     ws.part_small);
  const long long n1 = (long long)ld * HD;
  hipLaunchKernelGGL(sum_parts_kernel, dim3((unsigned)((n1 + 63) / 64)), dim3(256), 0, st, ws.part_w1, ws.chunks, n1,
                     n1, grad.w1);
  const long long ss = (long long)HD * HD + 2 * HD;
  hipLaunchKernelGGL(sum_parts_kernel, dim3((HD * HD + 63) / 64), dim3(256), 0, st, ws.part_small, ws.chunks_small,
                     (long long)HD * HD, ss, grad.w2);
  hipLaunchKernelGGL(sum_parts_kernel, dim3((HD + 63) / 64), dim3(256), 0, st, ws.part_small + HD * HD,
                     ws.chunks_small, (long long)HD, ss, grad.b1);
  hipLaunchKernelGGL(sum_parts_kernel, dim3((HD + 63) / 64), dim3(256), 0, st, ws.part_small + HD * HD + HD,
                     ws.chunks_small, (long long)HD, ss, grad.b2);
  return hipGetLastError();
}

// n (1 or 2) compressions of the same shape; with the MLP they share one launch (grid.y).
template <typename T, int HD>
hipError_t compress_impl(const Dims& D, const CompressJob* jobs, int n, const uint8_t* valid, hipStream_t st) {
  const long long rows = D.cmp_rows();
  if (D.pool == 1) {
    const long long tot = rows * HD;
    for (int i = 0; i < n; ++i)
      hipLaunchKernelGGL(mean_pool_kernel<T>, dim3((unsigned)((tot + 255) / 256)), dim3(256), 0, st,
                         (const T*)jobs[i].x, valid, D.H, D.N, D.l, HD, rows, jobs[i].out, (T*)jobs[i].out_lp,
                         jobs[i].lp_scale);
    return hipGetLastError();
  }
  const int ld = D.l * HD;
  MlpFwdJob mj[2];
  for (int i = 0; i < n; ++i) {
    const CompressJob& c = jobs[i];
    hipLaunchKernelGGL(transpose_w1_kernel<T>, dim3((ld * HD + 255) / 256), dim3(256), 0, st, c.phi.w1, ld, HD,
                       (T*)c.w1t_ws);
    mj[i] = MlpFwdJob{c.x, c.w1t_ws, c.phi.b1, c.phi.w2, c.phi.b2, c.out, c.pre, c.out_lp, c.lp_scale};
  }
  if (n == 1) mj[1] = mj[0];
  const long long per_wg = (long long)kWaves * 16 * kRB;
  const unsigned grid = (unsigned)((rows + per_wg - 1) / per_wg);
  hipLaunchKernelGGL((mlp_fwd_kernel<T, HD>), dim3(grid, (unsigned)n), dim3(kWaves * 64), 0, st, valid, D.H, D.N, D.l,
                     rows, mj[0], mj[1]);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_block_valid(const Dims& D, const uint8_t* valid, uint8_t* cvalid, hipStream_t st) {
  const int total = D.B * (D.N / D.l);
  hipLaunchKernelGGL(block_valid_kernel, dim3((total + 255) / 256), dim3(256), 0, st, valid, total, D.l, cvalid);
  return hipGetLastError();
}

int mlp_bwd_chunks_small(const Dims& D) {
  const long long rows = D.cmp_rows();
  long long c = rows / 128;
  if (c < 1) c = 1;
  if (c > 256) c = 256;
  return (int)c;
}

int mlp_bwd_chunks(const Dims& D) {
  const long long rows = D.cmp_rows();
  long long c = rows / 512;
  if (c < 1) c = 1;
  if (c > 64) c = 64;
  return (int)c;
}

hipError_t launch_compress_bwd(const Dims& D, const void* x, const uint8_t* valid, const Mlp& phi, const float* pre,
                               const float* dy, float* dx_accum, const MlpGrad& grad, const MlpBwdWs& ws,
                               hipStream_t st) {
  return BSA_DISPATCH(compress_bwd_impl, D, x, valid, phi, pre, dy, dx_accum, grad, ws, st);
}

hipError_t launch_compress_fwd(const Dims& D, const CompressJob* jobs, int n, const uint8_t* valid, hipStream_t st) {
  if (n < 1 || n > 2) return hipErrorInvalidValue;
  if (D.bf16)
    return D.d == 64 ? compress_impl<bf16_t, 64>(D, jobs, n, valid, st) : compress_impl<bf16_t, 32>(D, jobs, n, valid, st);
  return D.d == 64 ? compress_impl<float, 64>(D, jobs, n, valid, st) : compress_impl<float, 32>(D, jobs, n, valid, st);
}

}  // namespace bsa
