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
// four lists of each group are merged in registers at the end.
// Scores keep f32 accuracy so that rankings match the float64 definition except where two
// scores are closer than f32 rounding: each f32 operand is split into three bf16 parts
// (x = hi + mid + lo up to 2^-27 |x|) and a score is the f32 sum of the six products
// whose weight reaches 2^-16 (hi hi, hi mid, mid hi, hi lo, lo hi, mid mid), each exact in
// the bf16 matrix cores: about the error of an f32 product, at 6 bf16 MFMAs per 32-wide
// slice instead of 8 f32 ones per 4-wide slice.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "attn_common.hpp"

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

// Inverse of ordered_bits (the score of a key's upper word).
__device__ __forceinline__ float key_score(uint64_t key) {
  const uint32_t b = (uint32_t)(key >> 32);
  return __uint_as_float((b & 0x80000000u) ? (b & 0x7FFFFFFFu) : ~b);
}

// Insert x into the descending list (keys are unique, x > lst[K - 1]): every entry compares
// with x independently, then each slot keeps its entry, takes x, or takes its upper
// neighbour (slots are rewritten from the bottom, so the neighbour is still the old one).
template <int K>
__device__ __forceinline__ void topk_insert(uint64_t (&lst)[K], uint64_t x) {
  bool gt[K];
#pragma unroll
  for (int t = 0; t < K; ++t) gt[t] = lst[t] > x;
#pragma unroll
  for (int t = K - 1; t >= 1; --t) lst[t] = gt[t] ? lst[t] : (gt[t - 1] ? x : lst[t - 1]);
  lst[0] = gt[0] ? lst[0] : x;
}

// The group's four lanes L, L^16, L^32, L^48 exchange through gfx950's VALU lane swaps
// (no LDS traffic). With both operands holding x, v_permlane16_swap returns the values of
// the even and the odd 16-lane row of the lane's row pair, v_permlane32_swap those of the
// lower and the upper half; min and max are symmetric, so either order serves.
__device__ __forceinline__ void swap16_u64(uint64_t x, uint64_t& a, uint64_t& b) {
  const auto lo = __builtin_amdgcn_permlane16_swap((uint32_t)x, (uint32_t)x, false, false);
  const auto hi = __builtin_amdgcn_permlane16_swap((uint32_t)(x >> 32), (uint32_t)(x >> 32), false, false);
  a = ((uint64_t)hi[0] << 32) | lo[0];
  b = ((uint64_t)hi[1] << 32) | lo[1];
}
__device__ __forceinline__ void swap32_u64(uint64_t x, uint64_t& a, uint64_t& b) {
  const auto lo = __builtin_amdgcn_permlane32_swap((uint32_t)x, (uint32_t)x, false, false);
  const auto hi = __builtin_amdgcn_permlane32_swap((uint32_t)(x >> 32), (uint32_t)(x >> 32), false, false);
  a = ((uint64_t)hi[0] << 32) | lo[0];
  b = ((uint64_t)hi[1] << 32) | lo[1];
}
__device__ __forceinline__ uint64_t group_min_u64(uint64_t x) {
  uint64_t a, b;
  swap16_u64(x, a, b);
  x = a < b ? a : b;
  swap32_u64(x, a, b);
  return a < b ? a : b;
}
__device__ __forceinline__ uint64_t group_max_u64(uint64_t x) {
  uint64_t a, b;
  swap16_u64(x, a, b);
  x = a > b ? a : b;
  swap32_u64(x, a, b);
  return a > b ? a : b;
}
// x of the lanes r, r + 16, r + 32, r + 48 (r = L mod 16), in that order
__device__ __forceinline__ void group_gather(int x, int (&out)[4]) {
  const auto p = __builtin_amdgcn_permlane16_swap((uint32_t)x, (uint32_t)x, false, false);
  const auto e = __builtin_amdgcn_permlane32_swap(p[0], p[0], false, false);   // rows 0, 2
  const auto o = __builtin_amdgcn_permlane32_swap(p[1], p[1], false, false);   // rows 1, 3
  out[0] = (int)e[0];
  out[1] = (int)o[0];
  out[2] = (int)e[1];
  out[3] = (int)o[1];
}

// Pooled queries (Eq. 11): q_p = (1/g) * sum of the group's real queries, one thread per
// (group, channel); consecutive threads read consecutive channels of each query row.
template <typename T, int HD>
__global__ void pool_q_kernel(const T* q, const uint8_t* valid, int H, int N, int g, long long total, float* qpool) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int c = (int)(i % HD);
  const long long gp = i / HD;             // (b*H + h) * (N/g) + p
  const int ngroups = N / g;
  const long long bh = gp / ngroups;
  const int p = (int)(gp % ngroups);
  const int b = (int)(bh / H);
  const T* qr = q + ((size_t)bh * N + (size_t)p * g) * HD + c;
  const uint8_t* vb = valid ? valid + (size_t)b * N + (size_t)p * g : nullptr;
  float s = 0.f;
#pragma unroll 8
  for (int t = 0; t < g; ++t)
    if (vb == nullptr || vb[t]) s += to_f32<T>(qr[(size_t)t * HD]);
  qpool[i] = s / (float)g;
}

// hi = bf16(x), mid = bf16(x - hi), lo = bf16(x - hi - mid) (the differences are exact in
// f32); eight elements per thread.
__device__ __forceinline__ void split3(const float* x, bf16x8& hi, bf16x8& mid, bf16x8& lo) {
  float h[8], md[8], lw[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float a = x[e];
    const float ah = bf2f(f2bf(a));
    const float r1 = a - ah;
    const float am = bf2f(f2bf(r1));
    h[e] = ah;
    md[e] = am;
    lw[e] = r1 - am;
  }
  hi = make_chunk<bf16_t>(h);
  mid = make_chunk<bf16_t>(md);
  lo = make_chunk<bf16_t>(lw);
}

__global__ void __launch_bounds__(256) split3_kernel(const float* __restrict__ x, long long n8,
                                                     bf16_t* __restrict__ hi, bf16_t* __restrict__ mid,
                                                     bf16_t* __restrict__ lo) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= n8) return;
  const f32x8 v = load_chunk(x + 8 * i);
  float a[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) a[e] = v[e];
  bf16x8 h, m, l;
  split3(a, h, m, l);
  *reinterpret_cast<bf16x8*>(hi + 8 * i) = h;
  *reinterpret_cast<bf16x8*>(mid + 8 * i) = m;
  *reinterpret_cast<bf16x8*>(lo + 8 * i) = l;
}

template <typename T, int HD, int K, int R>
__global__ void __launch_bounds__(kWaves * 64) select_kernel(const float* qpool, const bf16_t* kplanes,
                                                             const uint8_t* cvalid, int H, int N, int l, int ls,
                                                             int m, int g, int mask_own, int kk, int* sel) {
  constexpr int NCH = HD / 32;
  constexpr int KT = 64;        // compressed tokens per staged tile
  constexpr int GW = 16 * kWaves;   // groups per workgroup
  // the three bf16 parts of a tile of compressed keys, double-buffered (distinct objects)
  __shared__ __attribute__((aligned(16))) bf16_t kh0[KT * HD], km0[KT * HD], kl0[KT * HD];
  __shared__ __attribute__((aligned(16))) bf16_t kh1[KT * HD], km1[KT * HD], kl1[KT * HD];
  __shared__ uint8_t cv0[KT], cv1[KT];
  __shared__ uint32_t av0, av1;   // 1: every compressed token of the staged tile is real
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15, j = lane >> 4;
  const int ngroups = N / g;
  const int bh = blockIdx.y;
  const int b = bh / H;
  const int p0 = blockIdx.x * GW;
  const int ntok = N / l;
  const size_t plane = (size_t)gridDim.y * ntok * HD;   // elements of one part
  const bf16_t* ph = kplanes + (size_t)bh * ntok * HD;
  const uint8_t* cv = cvalid + (size_t)b * (N / l);

  // compressed-token tiles: the three parts moved by direct global->LDS loads; token
  // validity bytes are read before the tile loads (by wave 0: KT == 64), and a flag marks
  // tiles whose tokens are all real
  static_assert(KT == 64, "wave 0 reads the validity of one tile");
  auto issue = [&](int t0, bf16_t* dh, bf16_t* dm, bf16_t* dl, uint8_t* cd, uint32_t* ad) {
    uint8_t c = 0;
    if (threadIdx.x < KT) c = t0 + (int)threadIdx.x < ntok ? cv[t0 + threadIdx.x] : 0;
    dma_tile<HD, KT, kWaves>(dh, ph, t0, ntok, wid, lane);
    dma_tile<HD, KT, kWaves>(dm, ph + plane, t0, ntok, wid, lane);
    dma_tile<HD, KT, kWaves>(dl, ph + 2 * plane, t0, ntok, wid, lane);
    if (threadIdx.x < KT) cd[threadIdx.x] = c;
    if (wid == 0) {
      const uint64_t real = __builtin_amdgcn_ballot_w64(c != 0);
      if (lane == 0) *ad = real == ~0ull ? 1u : 0u;
    }
  };
  issue(0, kh0, km0, kl0, cv0, &av0);

  // pooled queries of this lane's group (B operand), in three bf16 parts
  const int pg = p0 + 16 * wid + r;
  const float* qpr = qpool + ((size_t)bh * ngroups + (pg < ngroups ? pg : 0)) * HD;
  bf16x8 qh[NCH], qm[NCH], ql[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const f32x8 v = load_chunk(qpr + 32 * c + 8 * j);
    float a[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) a[e] = v[e];
    split3(a, qh[c], qm[c], ql[c]);
  }

  const int my_group = p0 + 16 * wid + r;
  const int my_ball = (my_group * g) / m;
  // selection blocks of the group's own ball (excluded when mask_own)
  const int own_lo = mask_own ? my_ball * (m / ls) : -1;
  const int own_hi = mask_own ? own_lo + m / ls : -1;
  uint64_t lst[K];
#pragma unroll
  for (int t = 0; t < K; ++t) lst[t] = 0;
  // The group's four lanes each keep a list; the group needs only its k* best (k* <= K).
  // Each lane's K/4 best are all at least the smallest of the four lanes' (K/4)-th keys,
  // so the group already holds K >= k* keys at or above that value and no candidate below
  // it can enter the final k*: the lanes filter on it as well as on their own K-th key.

  auto step = [&](int t0, const bf16_t* th, const bf16_t* tm, const bf16_t* tl_, const uint8_t* ct,
                  const uint32_t* at, bf16_t* nh, bf16_t* nm, bf16_t* nl, uint8_t* cn, uint32_t* an) {
    vm_drain();
    __syncthreads();
    const bool all_real = *at != 0u;
    if (t0 + KT < ntok) issue(t0 + KT, nh, nm, nl, cn, an);
    const uint64_t gthr = group_min_u64(lst[K / 4 - 1]);
    const uint64_t thr = gthr > lst[K - 1] ? gthr : lst[K - 1];
    // candidates pass on their score first (a key above thr has a score >= thr's); the
    // exact key comparison is made for the candidate that is inserted
    const float thr_f = thr == 0 ? kNegInf : key_score(thr);
    // the tile's candidates of this lane (4 / R per 16-token sub-tile, ascending blocks),
    // as scores; -inf = none
    constexpr int NPS = 4 / R;
    constexpr int NCAND = (KT / 16) * NPS;
    const int blk0 = (t0 + 4 * j) / R;
    float cand[NCAND];
    // scores of the tile's 4 sub-tiles: independent MFMA chains, interleaved
    f32x4 accs[KT / 16];
#pragma unroll
    for (int st = 0; st < KT / 16; ++st) accs[st] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      bf16x8 ah[KT / 16], am[KT / 16], al[KT / 16];
#pragma unroll
      for (int st = 0; st < KT / 16; ++st) {   // row 16 st + r, dims 32 c + 8 j ..
        ah[st] = lds_row_chunk<HD>(th, 16 * st + r, 4 * c + j);
        am[st] = lds_row_chunk<HD>(tm, 16 * st + r, 4 * c + j);
        al[st] = lds_row_chunk<HD>(tl_, 16 * st + r, 4 * c + j);
      }
      // smaller terms first
#pragma unroll
      for (int st = 0; st < KT / 16; ++st) accs[st] = mma(al[st], qh[c], accs[st]);
#pragma unroll
      for (int st = 0; st < KT / 16; ++st) accs[st] = mma(ah[st], ql[c], accs[st]);
#pragma unroll
      for (int st = 0; st < KT / 16; ++st) accs[st] = mma(am[st], qm[c], accs[st]);
#pragma unroll
      for (int st = 0; st < KT / 16; ++st) accs[st] = mma(am[st], qh[c], accs[st]);
#pragma unroll
      for (int st = 0; st < KT / 16; ++st) accs[st] = mma(ah[st], qm[c], accs[st]);
#pragma unroll
      for (int st = 0; st < KT / 16; ++st) accs[st] = mma(ah[st], qh[c], accs[st]);
    }
    // branch-free per candidate; the validity bytes are read only for tiles with padding
    // (a wave-uniform choice)
    auto build = [&](auto with_valid) {
#pragma unroll
      for (int st = 0; st < KT / 16; ++st) {
        const f32x4 acc = accs[st];
        // lane holds scores of compressed tokens t0 + 16 st + 4j + i for group my_group
        const int tl = 16 * st + 4 * j;
        const bool in_range = t0 + 16 * st < ntok;
#pragma unroll
        for (int u = 0; u < NPS; ++u) {
          float sc = 0.f;
#pragma unroll
          for (int i = 0; i < R; ++i) sc += acc[u * R + i];
          sc *= 1.0f / (float)R;
          bool ok = in_range;
          if (decltype(with_valid)::value) {
            uint32_t any = 0;
#pragma unroll
            for (int i = 0; i < R; ++i) any |= ct[tl + u * R + i];
            ok = ok & (any != 0);
          }
          const int blk = blk0 + st * (16 / R) + u;
          ok = ok & !((blk >= own_lo) & (blk < own_hi)) & (sc >= thr_f);
          cand[st * NPS + u] = ok ? sc : kNegInf;
        }
      }
    };
    if (all_real)
      build(std::false_type{});
    else
      build(std::true_type{});
    // insert the qualifying candidates best first; the wave repeats only as many times as
    // its busiest lane needs (most candidates fall below the lane's current k-th key)
    for (;;) {
      float bs = kNegInf;
      int bi = 0;
#pragma unroll
      for (int t = 0; t < NCAND; ++t) {   // first maximum: the lowest block among equal scores
        const bool better = cand[t] > bs;
        bs = better ? cand[t] : bs;
        bi = better ? t : bi;
      }
      const uint64_t key = bs > kNegInf ? make_key(bs, blk0 + (bi / NPS) * (16 / R) + bi % NPS) : 0;
      const uint64_t lim = thr > lst[K - 1] ? thr : lst[K - 1];
      const bool take = key > lim;
      if (!__builtin_amdgcn_ballot_w64(take)) break;
      if (take) {
        topk_insert<K>(lst, key);
#pragma unroll
        for (int t = 0; t < NCAND; ++t) cand[t] = t == bi ? kNegInf : cand[t];
      } else {
#pragma unroll
        for (int t = 0; t < NCAND; ++t) cand[t] = kNegInf;
      }
    }
  };
  for (int t0 = 0; t0 < ntok; t0 += 2 * KT) {
    step(t0, kh0, km0, kl0, cv0, &av0, kh1, km1, kl1, cv1, &av1);
    if (t0 + KT < ntok) step(t0 + KT, kh1, km1, kl1, cv1, &av1, kh0, km0, kl0, cv0, &av0);
  }
  // merge: the 4 sorted lists of group r sit in lanes r, r + 16, r + 32, r + 48 (the wave's
  // 16 groups side by side). k* rounds of a 4-way merge: the group's best head (two
  // exchanges) is chosen and its owner drops it; lane j keeps the blocks of rounds
  // j, j + 4, ... (-1 once the lists run dry).
  int mine[4] = {-1, -1, -1, -1};
#pragma unroll
  for (int t = 0; t < K; ++t) {
    if (t >= kk) break;
    const uint64_t head = lst[0];
    const uint64_t w = group_max_u64(head);
    const bool pop = w != 0 && head == w;   // keys are unique: one lane of the group holds w
#pragma unroll
    for (int i = 0; i < K - 1; ++i) lst[i] = pop ? lst[i + 1] : lst[i];
    lst[K - 1] = pop ? 0 : lst[K - 1];
    const int blk = w == 0 ? -1 : (int)(0xFFFFFFFFu - (uint32_t)(w & 0xFFFFFFFFu));
    mine[t >> 2] = (t & 3) == j ? blk : mine[t >> 2];
  }
  // stored ascending with -1 in unused slots: each chosen block goes to its rank among the
  // group's (at most 16) chosen blocks, which every lane of the group gathers
  int all[16];
#pragma unroll
  for (int s4 = 0; s4 < 4; ++s4) {
    int g4[4];
    group_gather(mine[s4], g4);
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) all[4 * q4 + s4] = g4[q4];
  }
  int nsel = 0;
#pragma unroll
  for (int e = 0; e < 16; ++e) nsel += all[e] >= 0;
  const int p = p0 + 16 * wid + r;
  if (p < ngroups) {
    int* out = sel + ((size_t)bh * ngroups + p) * kk;
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
      const int v = mine[s4];
      if (v >= 0) {
        int rank = 0;
#pragma unroll
        for (int e = 0; e < 16; ++e) rank += (all[e] >= 0) & (all[e] < v);
        out[rank] = v;
      }
      const int slot = j + 4 * s4;
      if (slot < kk && slot >= nsel) out[slot] = -1;
    }
  }
}

template <typename T, int HD, int K>
hipError_t select_k(const Dims& D, const void* q, const uint8_t* valid, const float* kcmp, const uint8_t* cvalid,
                    int* sel, float* qpool, bool given, uint16_t* kplanes, hipStream_t st) {
  const long long total = (long long)D.B * D.H * (D.N / D.g) * HD;
  if (!given)
    hipLaunchKernelGGL((pool_q_kernel<T, HD>), dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, (const T*)q,
                       valid, D.H, D.N, D.g, total, qpool);
  const long long n8 = D.cmp_rows() * HD / 8;
  bf16_t* kp = reinterpret_cast<bf16_t*>(kplanes);
  hipLaunchKernelGGL(split3_kernel, dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, st, kcmp, n8, kp,
                     kp + D.cmp_rows() * HD, kp + 2 * D.cmp_rows() * HD);
  const int ngroups = D.N / D.g;
  dim3 grid((ngroups + 16 * kWaves - 1) / (16 * kWaves), D.B * D.H);
  const int R = D.ls / D.l;
  if (R == 1)
    hipLaunchKernelGGL((select_kernel<T, HD, K, 1>), grid, dim3(kWaves * 64), 0, st, (const float*)qpool, (const bf16_t*)kp,
                       cvalid, D.H, D.N, D.l, D.ls, D.m, D.g, D.mask_own, D.k, sel);
  else if (R == 2)
    hipLaunchKernelGGL((select_kernel<T, HD, K, 2>), grid, dim3(kWaves * 64), 0, st, (const float*)qpool, (const bf16_t*)kp,
                       cvalid, D.H, D.N, D.l, D.ls, D.m, D.g, D.mask_own, D.k, sel);
  else
    hipLaunchKernelGGL((select_kernel<T, HD, K, 4>), grid, dim3(kWaves * 64), 0, st, (const float*)qpool, (const bf16_t*)kp,
                       cvalid, D.H, D.N, D.l, D.ls, D.m, D.g, D.mask_own, D.k, sel);
  return hipGetLastError();
}

template <typename T, int HD>
hipError_t select_hd(const Dims& D, const void* q, const uint8_t* valid, const float* kcmp, const uint8_t* cvalid,
                     int* sel, float* qpool, bool given, uint16_t* kplanes, hipStream_t st) {
  if (D.k <= 4) return select_k<T, HD, 4>(D, q, valid, kcmp, cvalid, sel, qpool, given, kplanes, st);
  if (D.k <= 8) return select_k<T, HD, 8>(D, q, valid, kcmp, cvalid, sel, qpool, given, kplanes, st);
  return select_k<T, HD, 16>(D, q, valid, kcmp, cvalid, sel, qpool, given, kplanes, st);
}

}  // namespace

hipError_t launch_select_topk(const Dims& D, const void* q, const uint8_t* valid, const float* kcmp,
                              const uint8_t* cvalid, int* sel, float* qpool, bool given, uint16_t* kplanes,
                              hipStream_t st) {
  if (D.bf16)
    return D.d == 64 ? select_hd<bf16_t, 64>(D, q, valid, kcmp, cvalid, sel, qpool, given, kplanes, st)
                     : select_hd<bf16_t, 32>(D, q, valid, kcmp, cvalid, sel, qpool, given, kplanes, st);
  return D.d == 64 ? select_hd<float, 64>(D, q, valid, kcmp, cvalid, sel, qpool, given, kplanes, st)
                   : select_hd<float, 32>(D, q, valid, kcmp, cvalid, sel, qpool, given, kplanes, st);
}

}  // namespace bsa
