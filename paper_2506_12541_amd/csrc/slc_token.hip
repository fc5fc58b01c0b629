// Selection attention with per-token selection (g = 1: Eq. 6-8 without the grouping of
// Eq. 10-12). Every query has its own k* blocks, so no two queries of a 16-row MFMA tile
// share keys and the query-major form of the grouped kernels would gather k* l' keys per
// query. These kernels run block-major instead: the (query, slot) pairs are sorted by
// selected block (the same stable radix sort the tree uses), one workgroup owns one block
// of one head, keeps its l' keys in registers and walks the queries that selected it in
// tiles of 16 gathered rows.
//  - Forward: each (query, block) pair yields a partial softmax state (scaled max m, sum l,
//    unnormalised o) in float32; a merge pass combines the k* partials of each query in
//    slot order into its output row and LSE.
//  - Backward: per tile the workgroup recomputes S = Q K^T and dP = dO V^T, accumulates
//    dK^T and dV^T of its block in registers (read-modify-written once per block: no float
//    atomics), and writes each pair's dQ contribution; a merge pass adds the k* parts of
//    each query to dQ in slot order.
// bf16 storage only.
#include "common.hpp"
#include "kernels.hpp"
#include "attn_common.hpp"

namespace bsa {
namespace {

typedef short s16x4_t __attribute__((ext_vector_type(4)));

// 16x16x16 bf16 product: A = 4 bf16 of row L % 16, B = 4 bf16 of column L % 16, both at
// contraction index 4 (L / 16) + e.
__device__ __forceinline__ f32x4 mma16bb(uint2 a, uint2 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4_t, a), __builtin_bit_cast(s16x4_t, b), c,
                                                   0, 0, 0);
}
__device__ __forceinline__ f32x4 mma16bf(uint2 a, const float (&bv)[4], f32x4 c) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  bf16x4 y = {(__bf16)bv[0], (__bf16)bv[1], (__bf16)bv[2], (__bf16)bv[3]};
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4_t, a), __builtin_bit_cast(s16x4_t, y), c,
                                                   0, 0, 0);
}

// 4 elements of column `col` from rows r0 .. r0 + 3 of a row-major [*, HD] bf16 matrix.
template <int HD>
__device__ __forceinline__ uint2 gather_col4(const bf16_t* m, int r0, int col) {
  const uint32_t a = m[(size_t)r0 * HD + col], b = m[(size_t)(r0 + 1) * HD + col];
  const uint32_t c = m[(size_t)(r0 + 2) * HD + col], d = m[(size_t)(r0 + 3) * HD + col];
  return make_uint2(a | (b << 16), c | (d << 16));
}

// One (query, slot) pair per selected block of a real query: key = (b*H + h) * (N/l') +
// block, value = query * k* + slot; other slots get the sentinel key (sorted last).
__global__ void slc1_pairs_kernel(const int* sel, const uint8_t* valid, long long total, int kk, int H, int N,
                                  int nblk, uint32_t sentinel, uint32_t* keys, uint32_t* vals) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const long long row = i / kk;        // (b*H + h) * N + p
  const int s = (int)(i % kk);
  const int p = (int)(row % N);
  const long long bh = row / N;
  const int b = (int)(bh / H);
  const int id = sel[i];
  const bool ok = id >= 0 && (valid == nullptr || valid[(size_t)b * N + p] != 0);
  keys[i] = ok ? (uint32_t)(bh * nblk + id) : sentinel;
  vals[i] = (uint32_t)p * (uint32_t)kk + (uint32_t)s;
}

__global__ void fill_i32_kernel(int* x, long long n, int v) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) x[i] = v;
}

__global__ void seg_bounds1_kernel(const uint32_t* keys, long long total, uint32_t sentinel, int* seg_start,
                                   int* seg_end) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const uint32_t kx = keys[i];
  if (kx == sentinel) return;
  if (i == 0 || keys[i - 1] != kx) seg_start[kx] = (int)i;
  if (i == total - 1 || keys[i + 1] != kx) seg_end[kx] = (int)(i + 1);
}

// ---- forward: partial softmax states of every (query, block) pair ----
// S^T = K Q^T puts one query per accumulator column (lane % 16) and the block's keys on
// the rows, so the softmax reductions run over a lane's rows and its column's four lane
// groups, and P^T is already the B operand of O^T = V^T P^T. LO: the softmax states only
// (no V operand, no partial outputs), formed exactly as in the full launch.
template <int HD, int KBW, bool LO = false>
__global__ void __launch_bounds__(256) slc1_fwd_kernel(const bf16_t* q, const bf16_t* k, const bf16_t* v,
                                                       const uint8_t* valid_all, const uint32_t* vals,
                                                       const int* seg_start, const int* seg_end, int H, int N,
                                                       int ls, int kk, float sl2, float* opart, float2* mlpart) {
  constexpr int NCH = HD / 32, DB = HD / 16;
  typedef bf16x8 CT;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15, j = lane >> 4;
  const long long seg = blockIdx.x;
  const int nblk = N / ls;
  const long long bh = seg / nblk;
  const int blk = (int)(seg % nblk);
  const int b = (int)(bh / H);
  const int s0 = seg_start[seg], s1 = seg_end[seg];
  if (s1 <= s0) return;   // uniform over the workgroup
  const int key0 = blk * ls;
  const bf16_t* kh = k + ((size_t)bh * N + key0) * HD;
  const bf16_t* vh = v + ((size_t)bh * N + key0) * HD;
  const bf16_t* qh = q + (size_t)bh * N * HD;
  const uint8_t* val = valid_all ? valid_all + (size_t)b * N + key0 : nullptr;

  CT kf[KBW][NCH];   // A operand of S^T: row = key 16 kb + r
  uint2 vt[KBW][DB];  // A operand of O^T: row = dim 16 db + r, contraction = keys 16 kb + 4 j + e
  bool kok[KBW][4];   // keys 16 kb + 4 j + i (this lane's accumulator rows)
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) {
#pragma unroll
    for (int c = 0; c < NCH; ++c) kf[kb][c] = load_chunk(kh + (size_t)(16 * kb + r) * HD + 32 * c + 8 * j);
    if constexpr (!LO) {
#pragma unroll
      for (int db = 0; db < DB; ++db) vt[kb][db] = gather_col4<HD>(vh, 16 * kb + 4 * j, 16 * db + r);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) kok[kb][i] = val == nullptr || val[16 * kb + 4 * j + i] != 0;
  }

  const int nitems = (s1 - s0 + 15) / 16;
  // this lane's query of item `it`: its pair value and Q row (B operand of S^T)
  auto fetch = [&](int it, uint32_t& pv, CT (&qf)[NCH]) {
    const int pi = s0 + 16 * it + r;
    pv = pi < s1 ? vals[pi] : 0xFFFFFFFFu;
    const int p = pv == 0xFFFFFFFFu ? 0 : (int)(pv / (uint32_t)kk);
#pragma unroll
    for (int c = 0; c < NCH; ++c) qf[c] = load_chunk(qh + (size_t)p * HD + 32 * c + 8 * j);
  };
  uint32_t pv_n = 0;
  CT qf_n[NCH];
  if (wid < nitems) fetch(wid, pv_n, qf_n);
  for (int it = wid; it < nitems; it += 4) {
    const uint32_t pv = pv_n;
    CT qf[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) qf[c] = qf_n[c];
    if (it + 4 < nitems) fetch(it + 4, pv_n, qf_n);   // next item's rows in flight
    f32x4 st[KBW];
    float mx = kNegInf;
#pragma unroll
    for (int kb = 0; kb < KBW; ++kb) {
      st[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NCH; ++c) st[kb] = mma(kf[kb][c], qf[c], st[kb]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float x = kok[kb][i] ? st[kb][i] * sl2 : kNegInf;
        st[kb][i] = x;
        mx = fmaxf(mx, x);
      }
    }
    mx = col_max(mx);
    const float mref = mx == kNegInf ? 0.f : mx;
    float l = 0.f;
    f32x4 o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KBW; ++kb) {
      float pr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pr[i] = fast_exp2(st[kb][i] - mref);   // masked keys: exp2(-inf) = 0
        l += pr[i];
      }
      if constexpr (!LO) {
#pragma unroll
        for (int db = 0; db < DB; ++db) o[db] = mma16bf(vt[kb][db], pr, o[db]);
      }
    }
    l = col_sum(l);
    if (pv != 0xFFFFFFFFu) {
      const size_t pair = ((size_t)bh * N) * kk + pv;   // ((b*H + h) * N + p) * k* + slot
      if constexpr (!LO) {
        float* op = opart + pair * HD;
#pragma unroll
        for (int db = 0; db < DB; ++db)
          *reinterpret_cast<float4*>(op + 16 * db + 4 * j) = make_float4(o[db][0], o[db][1], o[db][2], o[db][3]);
      }
      if (j == 0) mlpart[pair] = make_float2(mx, l);
    }
  }
}

// Output row and LSE of each query from its k* partial states (slot order); padding rows
// and rows without any eligible key get zeros and LSE -inf. One thread per 4 columns;
// out == nullptr: the LSE only (one thread per row does the work).
template <typename T, int HD>
__global__ void slc1_merge_kernel(const float* opart, const float2* mlpart, const int* sel, const uint8_t* valid,
                                  int H, int N, int kk, long long rows, T* out, float* lse) {
  constexpr int PR = HD / 4;
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * PR) return;
  const long long row = i / PR;
  const int c = (int)(i % PR);
  const long long bh = row / N;
  const int n = (int)(row % N);
  const int b = (int)(bh / H);
  const bool ok = valid == nullptr || valid[(size_t)b * N + n] != 0;
  const int* srow = sel + row * kk;
  if (out == nullptr && c != 0) return;
  float M = kNegInf;
  if (ok)
    for (int s = 0; s < kk; ++s)
      if (srow[s] >= 0) {
        const float2 ml = mlpart[row * kk + s];
        if (ml.y > 0.f) M = fmaxf(M, ml.x);
      }
  float L = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  if (M != kNegInf)
    for (int s = 0; s < kk; ++s)
      if (srow[s] >= 0) {
        const float2 ml = mlpart[row * kk + s];
        if (ml.y > 0.f) {
          const float w = exp2f(ml.x - M);
          L += w * ml.y;
          if (out == nullptr) continue;
          const float4 op = *reinterpret_cast<const float4*>(opart + (row * kk + s) * HD + 4 * c);
          acc.x += w * op.x;
          acc.y += w * op.y;
          acc.z += w * op.z;
          acc.w += w * op.w;
        }
      }
  if (c == 0) lse[row] = L > 0.f ? (M + log2f(L)) * kLn2 : kNegInf;
  if (out == nullptr) return;
  const float inv = L > 0.f ? 1.0f / L : 0.f;
  T* po = out + row * HD + 4 * c;
  po[0] = from_f32<T>(acc.x * inv);
  po[1] = from_f32<T>(acc.y * inv);
  po[2] = from_f32<T>(acc.z * inv);
  po[3] = from_f32<T>(acc.w * inv);
}

// ---- backward: dK, dV of the block and each pair's dQ part ----
// S = Q K^T (queries on the accumulator rows, one key per column) as in the grouped
// key-major pass, so P and dS are the B operands of dV^T = dO^T P and dK^T = Q^T dS, with
// Q^T and dO^T from transpose reads of the tile's rows in LDS. dQ^T = K^T dS^T takes dS^T
// from a wave-private [query][key] LDS tile. A query's packed row terms reach the lanes
// whose accumulator rows hold it by shuffles.
template <int HD, int KBW>
__global__ void __launch_bounds__(256) slc1_bwd_kernel(const bf16_t* q, const bf16_t* k, const bf16_t* v,
                                                       const bf16_t* dout, const uint8_t* valid_all,
                                                       const uint32_t* vals, const int* seg_start,
                                                       const int* seg_end, const float4* t4, int H, int N, int ls,
                                                       int kk, float sl2, float scale, float* dk, float* dv,
                                                       float* dqpart) {
  constexpr int NCH = HD / 32, DB = HD / 16, LS = 16 * KBW;
  typedef bf16x8 CT;
  __shared__ __attribute__((aligned(16))) bf16_t qs_all[4][16 * HD];
  __shared__ __attribute__((aligned(16))) bf16_t ds_all[4][16 * HD];
  __shared__ __attribute__((aligned(16))) bf16_t ps_all[4][16 * LS];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15, j = lane >> 4;
  const long long seg = blockIdx.x;
  const int nblk = N / ls;
  const long long bh = seg / nblk;
  const int blk = (int)(seg % nblk);
  const int b = (int)(bh / H);
  const int s0 = seg_start[seg], s1 = seg_end[seg];
  if (s1 <= s0) return;   // uniform over the workgroup
  const int key0 = blk * ls;
  const bf16_t* kh = k + ((size_t)bh * N + key0) * HD;
  const bf16_t* vh = v + ((size_t)bh * N + key0) * HD;
  const bf16_t* qh = q + (size_t)bh * N * HD;
  const bf16_t* dh = dout + (size_t)bh * N * HD;
  const float4* th = t4 + (size_t)bh * N;
  const uint8_t* val = valid_all ? valid_all + (size_t)b * N + key0 : nullptr;
  bf16_t* qs = qs_all[wid];
  bf16_t* ds = ds_all[wid];
  bf16_t* ps = ps_all[wid];

  CT kf[KBW][NCH], vf[KBW][NCH];   // B operands of S and dP: column = key 16 kb + r
  uint2 kt[KBW][DB];               // A operand of dQ^T: row = dim 16 db + r, contraction = keys 16 kb + 4 j + e
  bool kok[KBW];
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) {
    kok[kb] = val == nullptr || val[16 * kb + r] != 0;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      kf[kb][c] = load_chunk(kh + (size_t)(16 * kb + r) * HD + 32 * c + 8 * j);
      vf[kb][c] = load_chunk(vh + (size_t)(16 * kb + r) * HD + 32 * c + 8 * j);
    }
#pragma unroll
    for (int db = 0; db < DB; ++db) kt[kb][db] = gather_col4<HD>(kh, 16 * kb + 4 * j, 16 * db + r);
  }
  f32x4 dka[KBW][DB], dva[KBW][DB];
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb)
#pragma unroll
    for (int db = 0; db < DB; ++db) { dka[kb][db] = f32x4{0.f, 0.f, 0.f, 0.f}; dva[kb][db] = dka[kb][db]; }

  const int nitems = (s1 - s0 + 15) / 16;
  // this lane's query of item `it` (row r of the tile): pair value, Q and dO rows, terms
  auto fetch = [&](int it, uint32_t& pv, CT (&aq)[NCH], CT (&ad)[NCH], float4& tq) {
    const int pi = s0 + 16 * it + r;
    pv = pi < s1 ? vals[pi] : 0xFFFFFFFFu;
    const int p = pv == 0xFFFFFFFFu ? 0 : (int)(pv / (uint32_t)kk);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      aq[c] = load_chunk(qh + (size_t)p * HD + 32 * c + 8 * j);
      ad[c] = load_chunk(dh + (size_t)p * HD + 32 * c + 8 * j);
    }
    tq = th[p];
  };
  uint32_t pv_n = 0;
  CT aq_n[NCH], ad_n[NCH];
  float4 tq_n = make_float4(0.f, 0.f, 0.f, 0.f);
  if (wid < nitems) fetch(wid, pv_n, aq_n, ad_n, tq_n);
  for (int it = wid; it < nitems; it += 4) {
    const uint32_t pv = pv_n;
    CT aq[NCH], ad[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) { aq[c] = aq_n[c]; ad[c] = ad_n[c]; }
    float4 tq = tq_n;
    if (it + 4 < nitems) fetch(it + 4, pv_n, aq_n, ad_n, tq_n);   // next item's rows in flight
    const bool live = pv != 0xFFFFFFFFu;
    if (!live) tq = make_float4(__builtin_huge_valf(), 0.f, 0.f, 0.f);   // P = 0 on padding rows
    // terms of the queries on this lane's accumulator rows (4 j + i), from lanes 4 j + i
    float cl[4], cg[4], cdv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      cl[i] = __shfl(tq.x, 4 * j + i, 64);
      cg[i] = __shfl(tq.y, 4 * j + i, 64);
      cdv[i] = __shfl(tq.z, 4 * j + i, 64);
    }
    // the tile's Q and dO rows into LDS (swizzled) for the transpose reads
    wave_sync();   // the previous item's reads of the wave's tiles are done
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      *reinterpret_cast<CT*>(qs + r * HD + 8 * ((4 * c + j) ^ swz<HD>(r))) = aq[c];
      *reinterpret_cast<CT*>(ds + r * HD + 8 * ((4 * c + j) ^ swz<HD>(r))) = ad[c];
    }
    wave_sync();
    uint2 aqt[DB], adt[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      aqt[db] = lds_tr4<HD>(qs, 0, 16 * db, lane);
      adt[db] = lds_tr4<HD>(ds, 0, 16 * db, lane);
    }
#pragma unroll
    for (int kb = 0; kb < KBW; ++kb) {
      f32x4 sv = f32x4{0.f, 0.f, 0.f, 0.f}, dp = sv;
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        sv = mma(aq[c], kf[kb][c], sv);
        dp = mma(ad[c], vf[kb][c], dp);
      }
      float pg[4], dsv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float pr = kok[kb] ? fast_exp2(__builtin_fmaf(sv[i], sl2, -cl[i])) : 0.f;
        pg[i] = pr;
        dsv[i] = pr * (dp[i] - cdv[i]);
        ps[(4 * j + i) * LS + 16 * kb + r] = f2bf(dsv[i]);
      }
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        dva[kb][db] = mma16bf(adt[db], pg, dva[kb][db]);
        dka[kb][db] = mma16bf(aqt[db], dsv, dka[kb][db]);
      }
    }
    wave_sync();   // dS^T tile written by the whole wave
    f32x4 dq[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) dq[db] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KBW; ++kb) {
      const uint2 bs = *reinterpret_cast<const uint2*>(ps + r * LS + 16 * kb + 4 * j);   // dS[query r][keys]
#pragma unroll
      for (int db = 0; db < DB; ++db) dq[db] = mma16bb(kt[kb][db], bs, dq[db]);
    }
    if (live) {
      float* pq = dqpart + (((size_t)bh * N) * kk + pv) * HD;
#pragma unroll
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<float4*>(pq + 16 * db + 4 * j) =
            make_float4(dq[db][0] * scale, dq[db][1] * scale, dq[db][2] * scale, dq[db][3] * scale);
    }
  }
  // fixed-order sum of the four waves' block gradients (wave 0 adds waves 1, 2, 3), then
  // one read-modify-write of the block's dK, dV rows
  float* red0 = reinterpret_cast<float*>(&qs_all[0][0]);
  float* red1 = reinterpret_cast<float*>(&ds_all[0][0]);
  static_assert(16 * HD * 4 <= 4 * 16 * HD * 2, "reduction buffer");
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) {
    for (int w = 1; w < 4; ++w) {
      __syncthreads();
      if (wid == w) {
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const int o = r * HD + 16 * db + 4 * j;
          *reinterpret_cast<f32x4*>(&red0[o]) = dka[kb][db];
          *reinterpret_cast<f32x4*>(&red1[o]) = dva[kb][db];
        }
      }
      __syncthreads();
      if (wid == 0) {
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const int o = r * HD + 16 * db + 4 * j;
          dka[kb][db] += *reinterpret_cast<const f32x4*>(&red0[o]);
          dva[kb][db] += *reinterpret_cast<const f32x4*>(&red1[o]);
        }
      }
    }
  }
  if (wid != 0) return;
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) {
    const size_t off = ((size_t)bh * N + key0 + 16 * kb + r) * HD;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      float* pk = dk + off + 16 * db + 4 * j;
      float* pvp = dv + off + 16 * db + 4 * j;
      const float4 ok4 = *reinterpret_cast<const float4*>(pk), ov4 = *reinterpret_cast<const float4*>(pvp);
      const f32x4 a = dka[kb][db], c = dva[kb][db];
      *reinterpret_cast<float4*>(pk) =
          make_float4(ok4.x + a[0] * scale, ok4.y + a[1] * scale, ok4.z + a[2] * scale, ok4.w + a[3] * scale);
      *reinterpret_cast<float4*>(pvp) = make_float4(ov4.x + c[0], ov4.y + c[1], ov4.z + c[2], ov4.w + c[3]);
    }
  }
}

// dQ += the k* parts of each real query, in slot order. One thread per 4 columns.
template <int HD>
__global__ void slc1_merge_dq_kernel(const float* dqpart, const int* sel, const uint8_t* valid, int H, int N, int kk,
                                     long long rows, float* dq) {
  constexpr int PR = HD / 4;
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * PR) return;
  const long long row = i / PR;
  const int c = (int)(i % PR);
  const long long bh = row / N;
  const int n = (int)(row % N);
  const int b = (int)(bh / H);
  if (valid != nullptr && valid[(size_t)b * N + n] == 0) return;
  const int* srow = sel + row * kk;
  float4 acc = *reinterpret_cast<const float4*>(dq + row * HD + 4 * c);
  for (int s = 0; s < kk; ++s)
    if (srow[s] >= 0) {
      const float4 d = *reinterpret_cast<const float4*>(dqpart + (row * kk + s) * HD + 4 * c);
      acc.x += d.x;
      acc.y += d.y;
      acc.z += d.z;
      acc.w += d.w;
    }
  *reinterpret_cast<float4*>(dq + row * HD + 4 * c) = acc;
}

template <int HD, int KBW>
void fwd_launch(const Dims& D, const bf16_t* q, const bf16_t* k, const bf16_t* v, const uint8_t* valid,
                const uint32_t* vals, const Slc1Ws& W, long long nseg, float sl2, bool lse_only, hipStream_t st) {
  if (lse_only)
    hipLaunchKernelGGL((slc1_fwd_kernel<HD, KBW, true>), dim3((unsigned)nseg), dim3(256), 0, st, q, k, v, valid,
                       vals, W.seg_start, W.seg_end, D.H, D.N, D.ls, D.k, sl2, W.part, (float2*)W.ml);
  else
    hipLaunchKernelGGL((slc1_fwd_kernel<HD, KBW>), dim3((unsigned)nseg), dim3(256), 0, st, q, k, v, valid, vals,
                       W.seg_start, W.seg_end, D.H, D.N, D.ls, D.k, sl2, W.part, (float2*)W.ml);
}

template <int HD, int KBW>
void bwd_launch(const Dims& D, const bf16_t* q, const bf16_t* k, const bf16_t* v, const bf16_t* dout,
                const uint8_t* valid, const uint32_t* vals, const Slc1Ws& W, const float4* t4, long long nseg,
                float sl2, float* dk, float* dv, hipStream_t st) {
  hipLaunchKernelGGL((slc1_bwd_kernel<HD, KBW>), dim3((unsigned)nseg), dim3(256), 0, st, q, k, v, dout, valid, vals,
                     W.seg_start, W.seg_end, t4, D.H, D.N, D.ls, D.k, sl2, D.scale, dk, dv, W.part);
}

}  // namespace

size_t slc1_pairs(const Dims& D) { return (size_t)D.B * D.H * D.N * D.k; }

hipError_t launch_slc1_csr(const Dims& D, const int* sel, const uint8_t* valid, const Slc1Ws& W, uint32_t** vals_out,
                           hipStream_t st) {
  const long long total = (long long)slc1_pairs(D);
  const int nblk = D.N / D.ls;
  const long long nseg = (long long)D.B * D.H * nblk;
  const uint32_t sentinel = (uint32_t)nseg;
  int bits = 1;
  while ((1ll << bits) <= (long long)sentinel) ++bits;
  const unsigned g1 = (unsigned)((total + 255) / 256), gs = (unsigned)((nseg + 255) / 256);
  hipLaunchKernelGGL(slc1_pairs_kernel, dim3(g1), dim3(256), 0, st, sel, valid, total, D.k, D.H, D.N, nblk, sentinel,
                     W.keys, W.vals);
  hipLaunchKernelGGL(fill_i32_kernel, dim3(gs), dim3(256), 0, st, W.seg_start, nseg, 0);
  hipLaunchKernelGGL(fill_i32_kernel, dim3(gs), dim3(256), 0, st, W.seg_end, nseg, 0);
  uint32_t* kout = nullptr;
  hipError_t e = launch_radix_sort_pairs(W.keys, W.vals, W.keys_tmp, W.vals_tmp, W.hist, total, bits, &kout, vals_out,
                                         st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(seg_bounds1_kernel, dim3(g1), dim3(256), 0, st, kout, total, sentinel, W.seg_start, W.seg_end);
  return hipGetLastError();
}

hipError_t launch_slc1_fwd(const Dims& D, const void* q, const void* k, const void* v, const uint8_t* valid,
                           const int* sel, const Slc1Ws& W, void* o, float* lse, hipStream_t st) {
  if (!D.bf16) return hipErrorInvalidValue;
  uint32_t* vals = nullptr;
  hipError_t e = launch_slc1_csr(D, sel, valid, W, &vals, st);
  if (e != hipSuccess) return e;
  const long long nseg = (long long)D.B * D.H * (D.N / D.ls);
  const float sl2 = D.scale * kLog2e;
  const bf16_t *qq = (const bf16_t*)q, *kk = (const bf16_t*)k, *vv = (const bf16_t*)v;
  const int kbw = D.ls / 16;
  if (D.d == 64) {
    if (kbw == 1) fwd_launch<64, 1>(D, qq, kk, vv, valid, vals, W, nseg, sl2, o == nullptr, st);
    else if (kbw == 2) fwd_launch<64, 2>(D, qq, kk, vv, valid, vals, W, nseg, sl2, o == nullptr, st);
    else fwd_launch<64, 4>(D, qq, kk, vv, valid, vals, W, nseg, sl2, o == nullptr, st);
  } else {
    if (kbw == 1) fwd_launch<32, 1>(D, qq, kk, vv, valid, vals, W, nseg, sl2, o == nullptr, st);
    else if (kbw == 2) fwd_launch<32, 2>(D, qq, kk, vv, valid, vals, W, nseg, sl2, o == nullptr, st);
    else fwd_launch<32, 4>(D, qq, kk, vv, valid, vals, W, nseg, sl2, o == nullptr, st);
  }
  const long long rows = D.rows();
  const long long nt = rows * (D.d / 4);
  const unsigned grid = (unsigned)((nt + 255) / 256);
  if (D.d == 64)
    hipLaunchKernelGGL((slc1_merge_kernel<bf16_t, 64>), dim3(grid), dim3(256), 0, st, W.part, (const float2*)W.ml,
                       sel, valid, D.H, D.N, D.k, rows, (bf16_t*)o, lse);
  else
    hipLaunchKernelGGL((slc1_merge_kernel<bf16_t, 32>), dim3(grid), dim3(256), 0, st, W.part, (const float2*)W.ml,
                       sel, valid, D.H, D.N, D.k, rows, (bf16_t*)o, lse);
  return hipGetLastError();
}

hipError_t launch_slc1_bwd(const Dims& D, const void* q, const void* k, const void* v, const void* dout,
                           const uint8_t* valid, const int* sel, const float4* t4, const Slc1Ws& W, float* dk,
                           float* dv, hipStream_t st) {
  if (!D.bf16) return hipErrorInvalidValue;
  const int tid = timing_begin("bwd.slc_csr", st);
  uint32_t* vals = nullptr;
  hipError_t e = launch_slc1_csr(D, sel, valid, W, &vals, st);
  timing_end(tid, st);
  if (e != hipSuccess) return e;
  const long long nseg = (long long)D.B * D.H * (D.N / D.ls);
  const float sl2 = D.scale * kLog2e;
  const bf16_t *qq = (const bf16_t*)q, *kk = (const bf16_t*)k, *vv = (const bf16_t*)v, *dd = (const bf16_t*)dout;
  const int kbw = D.ls / 16;
  const int tkv = timing_begin("bwd.slc_kv", st);
  if (D.d == 64) {
    if (kbw == 1) bwd_launch<64, 1>(D, qq, kk, vv, dd, valid, vals, W, t4, nseg, sl2, dk, dv, st);
    else if (kbw == 2) bwd_launch<64, 2>(D, qq, kk, vv, dd, valid, vals, W, t4, nseg, sl2, dk, dv, st);
    else bwd_launch<64, 4>(D, qq, kk, vv, dd, valid, vals, W, t4, nseg, sl2, dk, dv, st);
  } else {
    if (kbw == 1) bwd_launch<32, 1>(D, qq, kk, vv, dd, valid, vals, W, t4, nseg, sl2, dk, dv, st);
    else if (kbw == 2) bwd_launch<32, 2>(D, qq, kk, vv, dd, valid, vals, W, t4, nseg, sl2, dk, dv, st);
    else bwd_launch<32, 4>(D, qq, kk, vv, dd, valid, vals, W, t4, nseg, sl2, dk, dv, st);
  }
  timing_end(tkv, st);
  return hipGetLastError();
}

hipError_t launch_slc1_merge_dq(const Dims& D, const int* sel, const uint8_t* valid, const Slc1Ws& W, float* dq,
                                hipStream_t st) {
  const long long rows = D.rows();
  const unsigned grid = (unsigned)((rows * (D.d / 4) + 255) / 256);
  if (D.d == 64)
    hipLaunchKernelGGL((slc1_merge_dq_kernel<64>), dim3(grid), dim3(256), 0, st, W.part, sel, valid, D.H, D.N, D.k,
                       rows, dq);
  else
    hipLaunchKernelGGL((slc1_merge_dq_kernel<32>), dim3(grid), dim3(256), 0, st, W.part, sel, valid, D.H, D.N, D.k,
                       rows, dq);
  return hipGetLastError();
}

}  // namespace bsa
