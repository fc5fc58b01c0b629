// Group selection (Section 2.2, Eq. 10-12 with the importance scores of Eq. 6 and the
// top-k of Eq. 7): every contiguous group of g queries pools its real queries into
// q_p = (1/g) * sum q_t, scores every compressed key by the unscaled product <q_p, k_c>,
// scores each selection block of r = l'/l compressed blocks by the mean of their scores,
// excludes blocks of the group's own ball and blocks without a real token, and keeps the
// k* best blocks (higher score first, lower block index on equal scores), stored in
// ascending block order with -1 in unused slots.
//
// The score matrix (N/g x N/l per head) is never stored. One workgroup owns 16 groups of
// one head: the pooled queries sit in registers as the B operand of f32 MFMA tiles, the
// four waves stream disjoint 16-token slices of the compressed keys from L2, and every
// lane keeps a running top-k of (ordered score, ~index) 64-bit keys for its group. The
// 16 partial lists of each group are merged through LDS by wave-wide argmax rounds.
// Scores stay in f32 end to end so that rankings match the float64 definition except
// where two scores are closer than f32 rounding.
#include "common.hpp"
#include "kernels.hpp"

namespace bsa {
namespace {

constexpr int kWaves = 4;

__device__ __forceinline__ uint32_t ordered_bits(float x) {
  x = x + 0.0f;
  uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ uint64_t make_key(float score, int blk) {
  return ((uint64_t)ordered_bits(score) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)blk);
}

template <int K>
__device__ __forceinline__ void topk_insert(uint64_t (&lst)[K], uint64_t x) {
  if (x <= lst[K - 1]) return;
#pragma unroll
  for (int t = 0; t < K; ++t) {
    uint64_t hi = lst[t] > x ? lst[t] : x;
    x = lst[t] > x ? x : lst[t];
    lst[t] = hi;
  }
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t x, int o) {
  uint32_t lo = (uint32_t)x, hi = (uint32_t)(x >> 32);
  lo = __shfl_xor(lo, o, 64);
  hi = __shfl_xor(hi, o, 64);
  return ((uint64_t)hi << 32) | lo;
}

template <typename T, int HD, int K, int R>
__global__ void __launch_bounds__(kWaves * 64) select_kernel(const T* q, const uint8_t* valid, const float* kcmp,
                                                             const uint8_t* cvalid, int H, int N, int l, int ls,
                                                             int m, int g, int mask_own, int kk, int* sel) {
  constexpr int NCH = HD / 32;
  __shared__ float qp[16][HD + 4];
  __shared__ uint64_t part[16][kWaves * 4 * K];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15, j = lane >> 4;
  const int ngroups = N / g;
  const int bh = blockIdx.y;
  const int b = bh / H;
  const int p0 = blockIdx.x * 16;
  const T* qh = q + (size_t)bh * N * HD;
  const float* kh = kcmp + (size_t)bh * (N / l) * HD;
  const uint8_t* vb = valid ? valid + (size_t)b * N : nullptr;
  const uint8_t* cv = cvalid + (size_t)b * (N / l);

  // pooled queries (Eq. 11) over the group's real queries
  for (int e = threadIdx.x; e < 16 * HD; e += blockDim.x) {
    int gi = e / HD, c = e % HD;
    int p = p0 + gi;
    float s = 0.f;
    if (p < ngroups) {
      for (int t = 0; t < g; ++t) {
        int tok = p * g + t;
        if (vb == nullptr || vb[tok]) s += to_f32<T>(qh[(size_t)tok * HD + c]);
      }
    }
    qp[gi][c] = s / (float)g;
  }
  __syncthreads();
  f32x8 bq[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int e = 0; e < 8; ++e) bq[c][e] = qp[r][32 * c + 8 * j + e];

  const int my_group = p0 + r;
  const int my_ball = (my_group * g) / m;
  uint64_t lst[K];
#pragma unroll
  for (int t = 0; t < K; ++t) lst[t] = 0;

  const int ntok = N / l;
  for (int tb = wid; tb < ntok / 16; tb += kWaves) {
    const float* kr = kh + (size_t)(tb * 16 + r) * HD;
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NCH; ++c) acc = mma(load_chunk(kr + 32 * c + 8 * j), bq[c], acc);
    // lane holds scores of compressed tokens tb*16 + 4j + i for group my_group
    const int t0 = tb * 16 + 4 * j;
#pragma unroll
    for (int u = 0; u < 4 / R; ++u) {
      float s = 0.f;
      bool ok = false;
#pragma unroll
      for (int i = 0; i < R; ++i) {
        s += acc[u * R + i];
        ok |= cv[t0 + u * R + i] != 0;
      }
      s *= 1.0f / (float)R;
      const int blk = (t0 + u * R) / R;
      if (mask_own && (blk * ls) / m == my_ball) ok = false;
      if (ok) topk_insert<K>(lst, make_key(s, blk));
    }
  }
  // partial lists -> LDS
#pragma unroll
  for (int t = 0; t < K; ++t) part[r][(wid * 4 + j) * K + t] = lst[t];
  __syncthreads();
  // merge: wave w finalises groups w, w+4, ...
  constexpr int NC = kWaves * 4 * K;  // candidates per group
  for (int gi = wid; gi < 16; gi += kWaves) {
    uint64_t cand[(NC + 63) / 64];
#pragma unroll
    for (int u = 0; u < (NC + 63) / 64; ++u) {
      int idx = u * 64 + lane;
      cand[u] = idx < NC ? part[gi][idx] : 0;
    }
    int mine = -1;
    for (int t = 0; t < kk; ++t) {
      uint64_t best = 0;
      int bu = 0;
#pragma unroll
      for (int u = 0; u < (NC + 63) / 64; ++u)
        if (cand[u] > best) { best = cand[u]; bu = u; }
      uint64_t w = best;
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        uint64_t y = shfl_xor_u64(w, o);
        w = y > w ? y : w;
      }
      if (w == 0) break;
      if (best == w) cand[bu] = 0;   // keys are unique: exactly one lane holds w
      if (lane == t) mine = (int)(0xFFFFFFFFu - (uint32_t)(w & 0xFFFFFFFFu));
    }
    // ascending order of the chosen blocks: rank among lanes < K
    const int p = p0 + gi;
    int rank = 0;
    for (int t = 0; t < kk; ++t) {
      int other = __shfl(mine, t, 64);
      if (other >= 0 && mine >= 0 && (other < mine)) ++rank;
    }
    int nsel = 0;
    for (int t = 0; t < kk; ++t) nsel += __shfl(mine, t, 64) >= 0;
    if (p < ngroups && lane < kk) {
      int* out = sel + ((size_t)bh * ngroups + p) * kk;
      if (mine >= 0) out[rank] = mine;
      if (lane >= nsel) out[lane] = -1;
    }
  }
}

template <typename T, int HD, int K>
hipError_t select_k(const Dims& D, const void* q, const uint8_t* valid, const float* kcmp, const uint8_t* cvalid,
                    int* sel, hipStream_t st) {
  const int ngroups = D.N / D.g;
  dim3 grid((ngroups + 15) / 16, D.B * D.H);
  const int R = D.ls / D.l;
  if (R == 1)
    hipLaunchKernelGGL((select_kernel<T, HD, K, 1>), grid, dim3(kWaves * 64), 0, st, (const T*)q, valid, kcmp, cvalid,
                       D.H, D.N, D.l, D.ls, D.m, D.g, D.mask_own, D.k, sel);
  else if (R == 2)
    hipLaunchKernelGGL((select_kernel<T, HD, K, 2>), grid, dim3(kWaves * 64), 0, st, (const T*)q, valid, kcmp, cvalid,
                       D.H, D.N, D.l, D.ls, D.m, D.g, D.mask_own, D.k, sel);
  else
    hipLaunchKernelGGL((select_kernel<T, HD, K, 4>), grid, dim3(kWaves * 64), 0, st, (const T*)q, valid, kcmp, cvalid,
                       D.H, D.N, D.l, D.ls, D.m, D.g, D.mask_own, D.k, sel);
  return hipGetLastError();
}

template <typename T, int HD>
hipError_t select_hd(const Dims& D, const void* q, const uint8_t* valid, const float* kcmp, const uint8_t* cvalid,
                     int* sel, hipStream_t st) {
  if (D.k <= 4) return select_k<T, HD, 4>(D, q, valid, kcmp, cvalid, sel, st);
  if (D.k <= 8) return select_k<T, HD, 8>(D, q, valid, kcmp, cvalid, sel, st);
  return select_k<T, HD, 16>(D, q, valid, kcmp, cvalid, sel, st);
}

}  // namespace

hipError_t launch_select_topk(const Dims& D, const void* q, const uint8_t* valid, const float* kcmp,
                              const uint8_t* cvalid, int* sel, hipStream_t st) {
  if (D.bf16)
    return D.d == 64 ? select_hd<bf16_t, 64>(D, q, valid, kcmp, cvalid, sel, st)
                     : select_hd<bf16_t, 32>(D, q, valid, kcmp, cvalid, sel, st);
  return D.d == 64 ? select_hd<float, 64>(D, q, valid, kcmp, cvalid, sel, st)
                   : select_hd<float, 32>(D, q, valid, kcmp, cvalid, sel, st);
}

}  // namespace bsa
