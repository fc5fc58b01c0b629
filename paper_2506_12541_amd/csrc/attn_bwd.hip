// Backward pass of the three attention branches and of the gate (Section 2.2, Eq. 3, 5,
// 8, 9). With dO_b = sigmoid(gamma_b) dO and per-row delta D_b = rowsum(dO_b * o_b), each
// branch is softmax attention, so with P = exp(S - LSE):
//     dP = dO_b V^T,  dS = P * (dP - D_b),  dQ = scale dS K,  dK = scale dS^T Q,  dV = P^T dO_b.
// The kernels fold the gate scale s = sigmoid(gamma_b) into the exponent: with
// E = s P = exp2(S log2e - (log2 LSE - log2 s)), dV = E^T dO and dS = E * (dO V^T - R_b),
// R_b = rowsum(dO * o_b) the unscaled delta, so no element needs a separate multiply by s.
// No gradient flows through the top-k selection (it is piecewise constant).
//
// Every gradient is produced without floating-point atomics, so results are
// deterministic: a query-major pass per branch accumulates dQ (forward layout: a lane
// owns one query, S^T = K Q^T), and a key-major pass accumulates dK and dV (a lane owns
// one key, S = Q K^T). The compressed branch splits its queries into chunks whose
// partial dK/dV are summed in a fixed order; the selection branch inverts the selected
// block lists (block -> groups, ascending) by a stable radix sort first.
#include <algorithm>
#include <limits>

#include "common.hpp"
#include "kernels.hpp"
#include "attn_common.hpp"

namespace bsa {
namespace {

__device__ __forceinline__ float sigmoidf(float x) { return 1.0f / (1.0f + __expf(-x)); }

// log2-domain LSE; rows without keys get +inf so that every probability is zero.
__device__ __forceinline__ float lse_log2(float lse) { return lse == -__builtin_huge_valf() ? __builtin_huge_valf() : lse * kLog2e; }

// ---- gate backward: R_b = rowsum(dO * o_b) per (b,h,n); dgamma_b = s'(gamma_b) sum_h R_b ----
// 8 lanes per row, each lane a 16-byte piece per tensor; partial sums reduced by shuffles.
// The same pass packs each query row's terms for the attention passes (16 bytes per row
// and branch; the layout QTerms describes). In bf16 layers the compressed branch's first
// term is stored negated: its passes start each score MFMA from it (prescaled keys).
template <typename T>
__global__ void gate_bwd_rows_kernel(const T* dout, const T* ob, const float* oc, long long rows, int hd,
                                     const float* lse, const float* gate, int H, int N, float* R, float4* terms) {
  constexpr int EPV = 16 / (int)sizeof(T);
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long row = gid >> 3;
  const int part = (int)(gid & 7);
  const long long per = rows * hd;
  float acc[3] = {0.f, 0.f, 0.f};
  if (row < rows) {
    for (int c = part * EPV; c < hd; c += 8 * EPV) {
      const uint4 dv = *reinterpret_cast<const uint4*>(dout + row * hd + c);
      const T* dp = reinterpret_cast<const T*>(&dv);
#pragma unroll
      for (int br = 0; br < 3; br += 2) {   // ball and selection rows (storage type)
        const uint4 ov = *reinterpret_cast<const uint4*>(ob + (br / 2) * per + row * hd + c);
        const T* op = reinterpret_cast<const T*>(&ov);
#pragma unroll
        for (int e = 0; e < EPV; ++e) acc[br] += to_f32<T>(dp[e]) * to_f32<T>(op[e]);
      }
#pragma unroll
      for (int e = 0; e < EPV; e += 4) {    // compressed-branch rows (float32)
        const float4 f = *reinterpret_cast<const float4*>(oc + row * hd + c + e);
        acc[1] += to_f32<T>(dp[e]) * f.x + to_f32<T>(dp[e + 1]) * f.y + to_f32<T>(dp[e + 2]) * f.z +
                  to_f32<T>(dp[e + 3]) * f.w;
      }
    }
  }
#pragma unroll
  for (int br = 0; br < 3; ++br) {
    float x = acc[br];
    x += __shfl_xor(x, 1, 64);
    x += __shfl_xor(x, 2, 64);
    x += __shfl_xor(x, 4, 64);
    acc[br] = x;
  }
  if (row < rows && part == 0) {
    const long long b = row / ((long long)H * N), n = row % N;
#pragma unroll
    for (int br = 0; br < 3; ++br) {
      R[br * rows + row] = acc[br];
      const float sg = sigmoidf(gate[(b * N + n) * 3 + br]);
      const float l2 = lse_log2(lse[br * rows + row]);
      const float x = l2 - log2f(sg);
      terms[br * rows + row] = make_float4(sizeof(T) == 2 && br == 1 ? -x : x, sg, acc[br], l2);
    }
  }
}

__global__ void gate_bwd_kernel(const float* R, const float* gate, const uint8_t* valid, int B, int H, int N,
                                float* dgate) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * N) return;
  int b = i / N, n = i % N;
  const long long rows = (long long)B * H * N;
#pragma unroll
  for (int br = 0; br < 3; ++br) {
    float sum = 0.f;
    if (valid == nullptr || valid[i])
      for (int h = 0; h < H; ++h) sum += R[br * rows + ((long long)b * H + h) * N + n];
    const float x = gate[(size_t)i * 3 + br];
    dgate[(size_t)i * 3 + br] = sigmoidf(x) * sigmoidf(-x) * sum;   // s(1-s) without cancellation
  }
}

// Group compression (Eq. 15), per coarse query: the copy's adjoint sums s_t dO_t over the
// real rows t of its block (s_t = sigmoid(gamma_cmp) of row t), kept in the storage type
// dO_c; its packed terms are (log2 LSE, 1, rowsum(dO_c * o_c), log2 LSE), the delta formed from
// the rounded dO_c the attention passes use and the float32 coarse output o_c, so that it
// equals their sum_j P_j dP_j to float32 rounding (near-uniform coarse softmaxes make dQ_c
// small next to either term). The log2 LSE is the one every real row of the block
// carries (+inf when the block has none). One thread per (coarse row, column); crows * hd
// is a multiple of 64, so every wave is whole and a row's hd lanes sit in one wave.
template <typename T>
__global__ void coarse_rows_bwd_kernel(const T* dout, const float4* t4b, const float* oc, const uint8_t* valid, int H,
                                       int N, int l, int hd, long long crows, T* doc, float4* t4c) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= crows * hd) return;
  const long long cr = i / hd;
  const int col = (int)(i % hd);
  const int nct = N / l;
  const long long bh = cr / nct;
  const int c = (int)(cr % nct);
  const int b = (int)(bh / H);
  const long long r0 = bh * N + (long long)c * l;
  const uint8_t* vb = valid ? valid + (size_t)b * N + (size_t)c * l : nullptr;
  float acc = 0.f, l2 = __builtin_huge_valf();
  for (int t = 0; t < l; ++t) {
    if (vb != nullptr && vb[t] == 0) continue;
    const float4 tt = t4b[r0 + t];
    acc += tt.y * to_f32<T>(dout[(r0 + t) * hd + col]);
    l2 = fminf(l2, tt.w);
  }
  const T dr = from_f32<T>(acc);
  doc[cr * hd + col] = dr;
  float dd = to_f32<T>(dr) * oc[cr * hd + col];
  for (int off = hd / 2; off > 0; off >>= 1) dd += __shfl_xor(dd, off, 64);
  if (col == 0) t4c[cr] = make_float4(sizeof(T) == 2 ? -l2 : l2, 1.f, dd, l2);   // negated in bf16, as above
}

template <typename T>
__global__ void cast_kernel(const float* x, long long n, float sc, T* y) {
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) y[i] = from_f32<T>(x[i] * sc);
}

__global__ void sum_chunks_kernel(const float* part, int nchunks, long long n, float* out) {
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float s = 0.f;
  for (int c = 0; c < nchunks; ++c) s += part[(long long)c * n + i];
  out[i] = s;
}

// Exact sign flip of 8 bf16 values (the sign bits). The backward passes multiply dO by -V
// (or -dO by V) so that the row term R of dS = P (dP - R) enters as the MFMA's accumulator
// input: the product then yields R - dP, and the sign moves into the final scale.
__device__ __forceinline__ bf16x8 neg_chunk(bf16x8 x) {
  uint4 u = __builtin_bit_cast(uint4, x);
  u.x ^= 0x80008000u;
  u.y ^= 0x80008000u;
  u.z ^= 0x80008000u;
  u.w ^= 0x80008000u;
  return __builtin_bit_cast(bf16x8, u);
}

// Per query row of one branch, packed (log2 LSE - log2 s, s, R, log2 LSE): s scales the
// row's dO (the branch gate sigmoid(gamma_b), or 1 for rows whose dO is already scaled),
// R = rowsum(dO * o_b) for the unscaled dO, so exp2(S log2e - x) is s P and the softmax
// gradient is s P (dO V^T - R). Rows without keys carry +inf in x and w. [B, H, N] float4.
// The compressed branch of bf16 layers stores -x instead (its keys come prescaled, so the
// score MFMA starting from -x yields the exponent S log2e - x directly).
struct QTerms {
  const float4* t4;
};

// ==== query-major pass, dense key sets (ball: own ball; compression: all tokens) ====
template <typename T, int HD, int QB, bool BALL, bool ADD>
__global__ void __launch_bounds__(256) dense_bwd_q_kernel(const T* q, const T* k, const T* v, const T* dout,
                                                          const uint8_t* kvalid_all, QTerms qt, int H, int N,
                                                          int nkeys_total, int m, float sl2, float scale, float* dq) {
  constexpr int NCH = HD / 32, DB = HD / 16;
  constexpr int KT = 64;   // keys per staged tile
  constexpr int KSTR = HD + 16 / (int)sizeof(T);
  constexpr int VSTR = KT + 4;
  typedef typename Chunk<T>::type CT;
  __shared__ __attribute__((aligned(16))) T ks[KT * KSTR];
  __shared__ __attribute__((aligned(16))) T vs[KT * KSTR];
  __shared__ __attribute__((aligned(16))) T kt[HD * VSTR];
  __shared__ __attribute__((aligned(16))) uint8_t kok[KT];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15, j = lane >> 4;
  const int b = blockIdx.z, h = blockIdx.y;
  const long long bh = (long long)b * H + h;
  const int q0 = blockIdx.x * (64 * QB);
  const int nkeys = BALL ? m : nkeys_total;
  const int key0 = BALL ? (q0 / m) * m : 0;
  const T* kh = k + (bh * nkeys_total + key0) * HD;
  const T* vh = v + (bh * nkeys_total + key0) * HD;
  const uint8_t* kval = kvalid_all ? kvalid_all + (size_t)b * nkeys_total + key0 : nullptr;
  const int wq0 = q0 + wid * 16 * QB;

  CT qf[QB][NCH], df[QB][NCH];
  float l2[QB], dd[QB], gs[QB];
  f32x4 acc[QB][DB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const long long row = bh * N + wq0 + 16 * qb + r;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      qf[qb][c] = load_chunk(q + row * HD + 32 * c + 8 * j);
      df[qb][c] = load_chunk(dout + row * HD + 32 * c + 8 * j);
    }
    const float4 t = qt.t4[row];
    l2[qb] = t.x;
    gs[qb] = t.y;
    dd[qb] = t.z;
#pragma unroll
    for (int db = 0; db < DB; ++db) acc[qb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  typedef TileIO<T, HD, KT> IO;
  uint4 kreg[IO::RV], vreg[IO::RV];
  typename IO::V4 treg[IO::TV][4];
  IO::load_rows(kreg, kh, 0, nkeys);
  IO::load_rows(vreg, vh, 0, nkeys);
  IO::load_tr(treg, kh, 0, nkeys);
  vm_drain();
  for (int t0 = 0; t0 < nkeys; t0 += KT) {
    __syncthreads();
    IO::store_rows(kreg, ks, KSTR);
    IO::store_rows(vreg, vs, KSTR);
    IO::store_tr(treg, kt, VSTR);
    if (threadIdx.x < KT) {
      const int key = t0 + threadIdx.x;
      kok[threadIdx.x] = key < nkeys && (kval == nullptr || kval[key]);
    }
    __syncthreads();
    if (t0 + KT < nkeys) {
      IO::load_rows(kreg, kh, t0 + KT, nkeys);
      IO::load_rows(vreg, vh, t0 + KT, nkeys);
      IO::load_tr(treg, kh, t0 + KT, nkeys);
    }
#pragma unroll
    for (int half = 0; half < KT / kKT; ++half) {
      const int h0 = half * kKT;
      if (t0 + h0 >= nkeys) break;
      constexpr int KB = kKT / 16;
      const bool all_ok = kval == nullptr && t0 + h0 + kKT <= nkeys;
      // key validity of the rows 4j+i of each key block, one 32-bit word per block
      uint32_t okw[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) okw[kb] = all_ok ? 0x01010101u : *reinterpret_cast<const uint32_t*>(&kok[h0 + kb * 16 + 4 * j]);
      f32x4 sv[QB][KB], dp[QB][KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          CT ak = load_chunk(&ks[(h0 + kb * 16 + r) * KSTR + 32 * c + 8 * j]);
          CT av = load_chunk(&vs[(h0 + kb * 16 + r) * KSTR + 32 * c + 8 * j]);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) {
            sv[qb][kb] = mma(ak, qf[qb][c], c == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : sv[qb][kb]);
            dp[qb][kb] = mma(av, df[qb][c], c == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : dp[qb][kb]);
          }
        }
      CT dsf[QB][KB / 2];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        float v8[KB][4];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float e = fast_exp2(__builtin_fmaf(sv[qb][kb][i], sl2, -l2[qb]));
            const float p = ((okw[kb] >> (8 * i)) & 1u) ? e : 0.f;
            v8[kb][i] = p * (dp[qb][kb][i] - dd[qb]);
          }
#pragma unroll
        for (int kp = 0; kp < KB / 2; ++kp) {
          float w8[8];
#pragma unroll
          for (int i = 0; i < 4; ++i) { w8[i] = v8[2 * kp][i]; w8[4 + i] = v8[2 * kp + 1][i]; }
          dsf[qb][kp] = make_chunk<T>(w8);
        }
      }
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int kp = 0; kp < KB / 2; ++kp) {
          CT a = load_4x2(&kt[(16 * db + r) * VSTR + h0 + 32 * kp + 4 * j]);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) acc[qb][db] = mma(a, dsf[qb][kp], acc[qb][db]);
        }
    }
  }
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const long long row = bh * N + wq0 + 16 * qb + r;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      float* dst = dq + row * HD + 16 * db + 4 * j;
      f32x4 val = acc[qb][db] * scale;
      if (ADD) {
        float4 old = *reinterpret_cast<float4*>(dst);
        val[0] += old.x; val[1] += old.y; val[2] += old.z; val[3] += old.w;
      }
      store4(dst, val, 1.0f);
    }
  }
}

// bf16 variant of the query-major pass: 64-key K and V tiles double-buffered in LDS (two
// distinct objects, loop unrolled by two) and filled by direct global->LDS loads; the K^T
// operand of the dQ product comes from transpose reads of the row-major K tile.
// MASK = false: every key is real and the key count is a multiple of the tile.
// PS: prescaled keys (the compressed tokens of bf16 layers): scores start from the stored
// -x and come out as exponents; dQ = dS K takes 1/log2(e) for the keys' extra factor.
template <int HD, int QB, bool BALL, bool ADD, bool MASK = true, bool PS = false>
__global__ void __launch_bounds__(256) dense_bwd_q_dma_kernel(const bf16_t* q, const bf16_t* k, const bf16_t* v,
                                                              const bf16_t* dout, const uint8_t* kvalid_all,
                                                              QTerms qt, int H, int N, int nkeys_total, int m,
                                                              float sl2, float scale, float* dq) {
  constexpr int NCH = HD / 32, DB = HD / 16;
  constexpr int KT = kKT;
  constexpr int KB = KT / 16;
  typedef bf16x8 CT;
  __shared__ __attribute__((aligned(16))) bf16_t ks0[KT * HD], ks1[KT * HD];
  __shared__ __attribute__((aligned(16))) bf16_t vs0[KT * HD], vs1[KT * HD];
  __shared__ __attribute__((aligned(16))) uint8_t ok0[KT], ok1[KT];
  const int lane = threadIdx.x & 63, wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 15, j = lane >> 4;
  const dim3 blk = xcd_grouped_block(BALL ? m / (64 * QB) : (int)gridDim.x);
  const int b = blk.z, h = blk.y;
  const long long bh = (long long)b * H + h;
  const int q0 = blk.x * (64 * QB);
  const int nkeys = BALL ? m : nkeys_total;
  const int key0 = BALL ? (q0 / m) * m : 0;
  const bf16_t* kh = k + (bh * nkeys_total + key0) * HD;
  const bf16_t* vh = v + (bh * nkeys_total + key0) * HD;
  const uint8_t* kval = kvalid_all ? kvalid_all + (size_t)b * nkeys_total + key0 : nullptr;
  const int wq0 = q0 + wid * 16 * QB;

  // key-validity bytes are read before the tile loads, so waiting for them does not
  // wait for the tile
  auto issue = [&](int t0, bf16_t* kd, bf16_t* vd, uint8_t* okd) {
    if constexpr (MASK) {
      uint8_t okv = 0;
      if (threadIdx.x < KT) {
        const int key = t0 + threadIdx.x;
        okv = key < nkeys && (kval == nullptr || kval[key]);
      }
      dma_tile<HD, KT, 4>(kd, kh, t0, nkeys, wid, lane);
      dma_tile<HD, KT, 4>(vd, vh, t0, nkeys, wid, lane);
      if (threadIdx.x < KT) okd[threadIdx.x] = okv;
    } else {   // whole tiles, every key real
      dma_tile_full<HD, KT, 4>(kd, kh + (size_t)t0 * HD, wid, lane);
      dma_tile_full<HD, KT, 4>(vd, vh + (size_t)t0 * HD, wid, lane);
    }
  };
  issue(0, ks0, vs0, ok0);

  // df holds -dO and rr the lane's R, so the dP product yields R - dO V^T
  CT qf[QB][NCH], df[QB][NCH];
  float l2[QB];
  f32x4 rr[QB], acc[QB][DB], s0[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const long long row = bh * N + wq0 + 16 * qb + r;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      qf[qb][c] = load_chunk(q + row * HD + 32 * c + 8 * j);
      df[qb][c] = neg_chunk(load_chunk(dout + row * HD + 32 * c + 8 * j));
    }
    const float4 t = qt.t4[row];   // log2 LSE - log2 s (negated with PS), s, R
    l2[qb] = t.x;
    rr[qb] = f32x4{t.z, t.z, t.z, t.z};
    s0[qb] = PS ? f32x4{t.x, t.x, t.x, t.x} : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int db = 0; db < DB; ++db) acc[qb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  auto step = [&](int t0, const bf16_t* kt, const bf16_t* vt, const uint8_t* ok, bf16_t* kn, bf16_t* vn,
                  uint8_t* okn) {
    vm_drain();          // this wave's loads of the tile have landed
    __syncthreads();     // ... and every wave's; the previous tile is no longer read
    if (t0 + KT < nkeys) issue(t0 + KT, kn, vn, okn);
    const bool all_ok = kval == nullptr && t0 + KT <= nkeys;
    // key validity of the rows 4j+i of each key block, one 32-bit word per block
    uint32_t okw[KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
      okw[kb] = all_ok ? 0x01010101u : *reinterpret_cast<const uint32_t*>(&ok[kb * 16 + 4 * j]);
    f32x4 sv[QB][KB], dp[QB][KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        CT ak = lds_row_chunk<HD>(kt, kb * 16 + r, 4 * c + j);
        CT av = lds_row_chunk<HD>(vt, kb * 16 + r, 4 * c + j);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          sv[qb][kb] = mma(ak, qf[qb][c], c == 0 ? s0[qb] : sv[qb][kb]);
          dp[qb][kb] = mma(av, df[qb][c], c == 0 ? rr[qb] : dp[qb][kb]);
        }
      }
    // dsf = P (R - dP) = -dS
    CT dsf[QB][KB / 2];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float v8[KB][4];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = PS ? fast_exp2(sv[qb][kb][i]) : fast_exp2(__builtin_fmaf(sv[qb][kb][i], sl2, -l2[qb]));
          const float p = !MASK || ((okw[kb] >> (8 * i)) & 1u) ? e : 0.f;
          v8[kb][i] = p * dp[qb][kb][i];
        }
#pragma unroll
      for (int kp = 0; kp < KB / 2; ++kp) {
        float w8[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) { w8[i] = v8[2 * kp][i]; w8[4 + i] = v8[2 * kp + 1][i]; }
        dsf[qb][kp] = make_chunk<bf16_t>(w8);
      }
    }
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int kp = 0; kp < KB / 2; ++kp) {
        CT a = lds_tr_chunk<HD>(kt, 32 * kp, 16 * db, lane);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) acc[qb][db] = mma(a, dsf[qb][kp], acc[qb][db]);
      }
  };
  for (int t0 = 0; t0 < nkeys; t0 += 2 * KT) {
    step(t0, ks0, vs0, ok0, ks1, vs1, ok1);
    if (t0 + KT < nkeys) step(t0 + KT, ks1, vs1, ok1, ks0, vs0, ok0);
  }
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const long long row = bh * N + wq0 + 16 * qb + r;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      float* dst = dq + row * HD + 16 * db + 4 * j;
      f32x4 val = acc[qb][db] * (PS ? -scale / sl2 : -scale);
      if (ADD) {
        float4 old = *reinterpret_cast<float4*>(dst);
        val[0] += old.x; val[1] += old.y; val[2] += old.z; val[3] += old.w;
      }
      store4(dst, val, 1.0f);
    }
  }
}

// ==== key-major pass, dense key sets: dK, dV of NW*32 keys per workgroup ====
// Queries are staged 64 at a time in LDS (row-major for the S and dP products, transposed
// for the dK^T and dV^T products); each wave owns 32 keys in registers.
constexpr int kQT = 64;
constexpr int kSlcLightItems = 256;   // selection dK/dV: blocks with more items get eight waves
constexpr int kSlcHeavyGroups = 256;  // persistent eight-wave workgroups of that second launch

template <typename T, int HD, int NW, bool BALL>
__global__ void __launch_bounds__(NW * 64) dense_bwd_kv_kernel(const T* q, const T* k, const T* v, const T* dout,
                                                               const uint8_t* kvalid_all, QTerms qt, int H, int N,
                                                               int nkeys_total, int m, int nchunks, float sl2,
                                                               float scale, float* dk_out, float* dv_out) {
  constexpr int NCH = HD / 32, DB = HD / 16;
  constexpr int QSTR = HD + 16 / (int)sizeof(T);
  constexpr int TSTR = kQT + 4;
  constexpr int KBW = 2;  // 16-key blocks per wave
  typedef typename Chunk<T>::type CT;
  __shared__ __attribute__((aligned(16))) T qs[kQT * QSTR];
  __shared__ __attribute__((aligned(16))) T ds_[kQT * QSTR];
  __shared__ __attribute__((aligned(16))) T qtr[HD * TSTR];
  __shared__ __attribute__((aligned(16))) T dtr[HD * TSTR];
  __shared__ __attribute__((aligned(16))) float l2s[kQT], dds[kQT], gss[kQT];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15, j = lane >> 4;
  const int bh = blockIdx.z;
  const int b = bh / H;
  const int chunk = blockIdx.y;
  const int key0 = blockIdx.x * (NW * 32);
  const int wk0 = key0 + wid * 32;
  int qbeg, qend;
  if (BALL) {
    qbeg = (key0 / m) * m;
    qend = qbeg + m;
  } else {
    const int per = N / nchunks;
    qbeg = chunk * per;
    qend = qbeg + per;
  }
  const T* qh = q + (size_t)bh * N * HD;
  const T* dh = dout + (size_t)bh * N * HD;
  const long long rowbase = (long long)bh * N;

  CT kf[KBW][NCH], vf[KBW][NCH];
  bool kok[KBW];
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) {
    const int key = wk0 + 16 * kb + r;
    kok[kb] = key < nkeys_total && (kvalid_all == nullptr || kvalid_all[(size_t)b * nkeys_total + key]);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      kf[kb][c] = zero_chunk(kf[kb][c]);
      vf[kb][c] = zero_chunk(vf[kb][c]);
      if (key < nkeys_total) {
        kf[kb][c] = load_chunk(k + ((size_t)bh * nkeys_total + key) * HD + 32 * c + 8 * j);
        vf[kb][c] = load_chunk(v + ((size_t)bh * nkeys_total + key) * HD + 32 * c + 8 * j);
      }
    }
  }
  f32x4 dka[KBW][DB], dva[KBW][DB];
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb)
#pragma unroll
    for (int db = 0; db < DB; ++db) { dka[kb][db] = f32x4{0.f, 0.f, 0.f, 0.f}; dva[kb][db] = dka[kb][db]; }

  // query tiles: row-major Q, dO and transposed Q^T, dO^T, prefetched one tile ahead
  typedef TileIO<T, HD, kQT, NW * 64> IO;
  uint4 qreg[IO::RV], dreg[IO::RV];
  typename IO::V4 qtreg[IO::TV][4], dtreg[IO::TV][4];
  float4 tv = make_float4(0.f, 0.f, 0.f, 0.f);
  auto fetch = [&](int t0) {
    IO::load_rows(qreg, qh, t0, N);
    IO::load_rows(dreg, dh, t0, N);
    IO::load_tr(qtreg, qh, t0, N);
    IO::load_tr(dtreg, dh, t0, N);
    if (threadIdx.x < kQT) {
      const long long row = rowbase + t0 + threadIdx.x;
      tv = qt.t4[row];
    }
  };
  fetch(qbeg);
  vm_drain();
  for (int t0 = qbeg; t0 < qend; t0 += kQT) {
    __syncthreads();
    IO::store_rows(qreg, qs, QSTR);
    IO::store_rows(dreg, ds_, QSTR);
    IO::store_tr(qtreg, qtr, TSTR);
    IO::store_tr(dtreg, dtr, TSTR);
    if (threadIdx.x < kQT) {
      l2s[threadIdx.x] = tv.x;
      gss[threadIdx.x] = tv.y;
      dds[threadIdx.x] = tv.z;
    }
    __syncthreads();
    if (t0 + kQT < qend) fetch(t0 + kQT);
#pragma unroll
    for (int qp = 0; qp < kQT / 32; ++qp) {
      f32x4 sv[2][KBW], dp[2][KBW];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int qb = 2 * qp + u;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          CT aq = load_chunk(&qs[(16 * qb + r) * QSTR + 32 * c + 8 * j]);
          CT ad = load_chunk(&ds_[(16 * qb + r) * QSTR + 32 * c + 8 * j]);
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) {
            sv[u][kb] = mma(aq, kf[kb][c], c == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : sv[u][kb]);
            dp[u][kb] = mma(ad, vf[kb][c], c == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : dp[u][kb]);
          }
        }
      }
      // lane holds queries 16qb + 4j + i for its key
      CT pf[KBW], sf[KBW];
      float a8[KBW][8], b8[KBW][8];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int qb = 2 * qp + u;
        const float4 L = *reinterpret_cast<const float4*>(&l2s[16 * qb + 4 * j]);
        const float4 Dd = *reinterpret_cast<const float4*>(&dds[16 * qb + 4 * j]);
        const float4 G = *reinterpret_cast<const float4*>(&gss[16 * qb + 4 * j]);
        const float lv[4] = {L.x, L.y, L.z, L.w}, dv4[4] = {Dd.x, Dd.y, Dd.z, Dd.w}, gv[4] = {G.x, G.y, G.z, G.w};
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float p = kok[kb] ? fast_exp2(__builtin_fmaf(sv[u][kb][i], sl2, -lv[i])) : 0.f;
            a8[kb][4 * u + i] = p;
            b8[kb][4 * u + i] = p * (dp[u][kb][i] - dv4[i]);
          }
      }
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) {
        pf[kb] = make_chunk<T>(a8[kb]);
        sf[kb] = make_chunk<T>(b8[kb]);
      }
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        CT ao = load_4x2(&dtr[(16 * db + r) * TSTR + 32 * qp + 4 * j]);
        CT aq = load_4x2(&qtr[(16 * db + r) * TSTR + 32 * qp + 4 * j]);
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
          dva[kb][db] = mma(ao, pf[kb], dva[kb][db]);
          dka[kb][db] = mma(aq, sf[kb], dka[kb][db]);
        }
      }
    }
  }
  // lane: key wk0 + 16kb + r, dims 16db + 4j + i
  const size_t out_base = (size_t)chunk * ((size_t)gridDim.z * nkeys_total * HD);
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) {
    const int key = wk0 + 16 * kb + r;
    if (key >= nkeys_total) continue;
    const size_t off = out_base + ((size_t)bh * nkeys_total + key) * HD;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      store4(dk_out + off + 16 * db + 4 * j, dka[kb][db], scale);
      store4(dv_out + off + 16 * db + 4 * j, dva[kb][db], 1.0f);
    }
  }
}

// bf16 variant of the key-major pass: 64-query tiles of Q, dO and the packed row terms
// double-buffered in LDS (two distinct objects, loop unrolled by two) and filled by direct
// global->LDS loads; the transposed operands of the dK^T and dV^T products come from
// transpose reads of the same row-major tiles.
// MASK = false: every key of the grid is real and in range (no per-key select).
// PS: prescaled keys (the compressed tokens of bf16 layers): scores start from the stored
// -x and come out as exponents (dK and dV do not involve the keys).
// KBW: 16-key blocks per wave (1 halves the registers: more waves for the HBM-bound ball pass).
// The unmasked compressed pass is held to 168 registers, three waves per SIMD instead of
// two: its MFMA pipe idles while a wave waits on its LDS reads and on its own results,
// and a third wave fills more of that (a few registers spill, outside the loop).
// LDS of the key-major pass: query and dO tiles and the row terms, double buffered
// (distinct objects, so that the compiler can tell in-flight loads into one buffer from
// reads of the other). The row terms are two arrays (log2 LSE - log2 s, and R) so that a
// lane reads the values of its four accumulator rows with one 16-byte load.
struct KvLds {
  bf16_t *qs0, *qs1, *ds0, *ds1;
  float *tx0, *tz0, *tx1, *tz1;
};
#define BSA_KV_LDS(L)                                                                      \
  __shared__ __attribute__((aligned(16))) bf16_t L##_qs0[kQT * HD], L##_qs1[kQT * HD];     \
  __shared__ __attribute__((aligned(16))) bf16_t L##_ds0[kQT * HD], L##_ds1[kQT * HD];     \
  __shared__ __attribute__((aligned(16))) float L##_tx0[kQT], L##_tz0[kQT], L##_tx1[kQT], \
      L##_tz1[kQT];                                                                        \
  const KvLds L{L##_qs0, L##_qs1, L##_ds0, L##_ds1, L##_tx0, L##_tz0, L##_tx1, L##_tz1}

struct KvArgs {
  const bf16_t *q, *k, *v, *dout;
  const uint8_t* kvalid_all;
  QTerms qt;
  int H, N, nkeys_total, m, nchunks;
  float sl2, scale;
  float *dk_out, *dv_out;
};

// One workgroup of the pass: `lin` is its linear id in a grid of shape `grid`.
template <int HD, int NW, bool BALL, bool MASK, bool PS, int KBW>
__device__ __forceinline__ void kv_dma_body(const KvLds& L, dim3 grid, unsigned lin, const KvArgs& a) {
  constexpr int NCH = HD / 32, DB = HD / 16;
  typedef bf16x8 CT;
  bf16_t *const qs0 = L.qs0, *const qs1 = L.qs1, *const ds0 = L.ds0, *const ds1 = L.ds1;
  float *const tx0 = L.tx0, *const tz0 = L.tz0, *const tx1 = L.tx1, *const tz1 = L.tz1;
  const bf16_t *const q = a.q, *const k = a.k, *const v = a.v, *const dout = a.dout;
  const uint8_t* const kvalid_all = a.kvalid_all;
  const QTerms qt = a.qt;
  const int H = a.H, N = a.N, nkeys_total = a.nkeys_total, m = a.m, nchunks = a.nchunks;
  const float sl2 = a.sl2, scale = a.scale;
  float *const dk_out = a.dk_out, *const dv_out = a.dv_out;
  const int lane = threadIdx.x & 63, wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 15, j = lane >> 4;
  const dim3 blk = xcd_grouped_block_at(lin, grid, BALL ? m / (NW * 16 * KBW) : (int)grid.x);
  const int bh = blk.z;
  const int b = bh / H;
  const int chunk = blk.y;
  const int key0 = blk.x * (NW * 16 * KBW);
  const int wk0 = key0 + wid * 16 * KBW;
  int qbeg, qend;
  if (BALL) {
    qbeg = (key0 / m) * m;
    qend = qbeg + m;
  } else {
    const int per = N / nchunks;
    qbeg = chunk * per;
    qend = qbeg + per;
  }
  const bf16_t* qh = q + (size_t)bh * N * HD;
  const bf16_t* dh = dout + (size_t)bh * N * HD;
  const float4* th = qt.t4 + (size_t)bh * N;

  auto issue = [&](int t0, bf16_t* qd, bf16_t* dd, float* txd, float* tzd) {
    dma_tile_full<HD, kQT, NW>(qd, qh + (size_t)t0 * HD, wid, lane);   // query tiles are whole (N % 64 == 0)
    dma_tile_full<HD, kQT, NW>(dd, dh + (size_t)t0 * HD, wid, lane);
    if (wid == NW - 1) {
      const float* t = reinterpret_cast<const float*>(th + t0 + lane);
      __builtin_amdgcn_global_load_lds(t, txd, 4, 0, 0);
      __builtin_amdgcn_global_load_lds(t + 2, tzd, 4, 0, 0);
    }
  };
  issue(qbeg, qs0, ds0, tx0, tz0);

  CT kf[KBW][NCH], vf[KBW][NCH];
  bool kok[KBW];
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) {
    const int key = wk0 + 16 * kb + r;
    kok[kb] = key < nkeys_total && (kvalid_all == nullptr || kvalid_all[(size_t)b * nkeys_total + key]);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      kf[kb][c] = zero_chunk(kf[kb][c]);
      vf[kb][c] = zero_chunk(vf[kb][c]);
      if (key < nkeys_total) {
        kf[kb][c] = load_chunk(k + ((size_t)bh * nkeys_total + key) * HD + 32 * c + 8 * j);
        vf[kb][c] = neg_chunk(load_chunk(v + ((size_t)bh * nkeys_total + key) * HD + 32 * c + 8 * j));
      }
    }
  }
  f32x4 dka[KBW][DB], dva[KBW][DB];
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb)
#pragma unroll
    for (int db = 0; db < DB; ++db) { dka[kb][db] = f32x4{0.f, 0.f, 0.f, 0.f}; dva[kb][db] = dka[kb][db]; }

  auto step = [&](int t0, const bf16_t* qs, const bf16_t* ds, const float* tx, const float* tz, bf16_t* qn,
                  bf16_t* dn, float* txn, float* tzn) {
    vm_drain();          // this wave's loads of the tile have landed
    __syncthreads();     // ... and every wave's; the previous tile is no longer read
    if (t0 + kQT < qend) issue(t0 + kQT, qn, dn, txn, tzn);
#pragma unroll
    for (int qp = 0; qp < kQT / 32; ++qp) {
      // lane holds queries 16qb + 4j + i for its key; dp = R - dO V^T (vf holds -V)
      f32x4 sv[2][KBW], dp[2][KBW], lx[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int qb = 2 * qp + u;
        lx[u] = *reinterpret_cast<const f32x4*>(&tx[16 * qb + 4 * j]);   // log2 LSE - log2 s (negated with PS)
        const f32x4 rz = *reinterpret_cast<const f32x4*>(&tz[16 * qb + 4 * j]);
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          CT aq = lds_row_chunk<HD>(qs, 16 * qb + r, 4 * c + j);
          CT ad = lds_row_chunk<HD>(ds, 16 * qb + r, 4 * c + j);
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) {
            sv[u][kb] = mma(aq, kf[kb][c], c == 0 ? (PS ? lx[u] : f32x4{0.f, 0.f, 0.f, 0.f}) : sv[u][kb]);
            dp[u][kb] = mma(ad, vf[kb][c], c == 0 ? rz : dp[u][kb]);
          }
        }
      }
      // a8 = P, b8 = P (R - dP) = -dS
      float a8[KBW][8], b8[KBW][8];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) {
            const float e = PS ? fast_exp2(sv[u][kb][i]) : fast_exp2(__builtin_fmaf(sv[u][kb][i], sl2, -lx[u][i]));
            const float p = !MASK || kok[kb] ? e : 0.f;
            a8[kb][4 * u + i] = p;
            b8[kb][4 * u + i] = p * dp[u][kb][i];
          }
        }
      }
      CT pf[KBW], sf[KBW];
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) {
        pf[kb] = make_chunk<bf16_t>(a8[kb]);
        sf[kb] = make_chunk<bf16_t>(b8[kb]);
      }
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        CT ao = lds_tr_chunk<HD>(ds, 32 * qp, 16 * db, lane);
        CT aq = lds_tr_chunk<HD>(qs, 32 * qp, 16 * db, lane);
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
          dva[kb][db] = mma(ao, pf[kb], dva[kb][db]);
          dka[kb][db] = mma(aq, sf[kb], dka[kb][db]);
        }
      }
    }
  };
  for (int t0 = qbeg; t0 < qend; t0 += 2 * kQT) {
    step(t0, qs0, ds0, tx0, tz0, qs1, ds1, tx1, tz1);
    if (t0 + kQT < qend) step(t0 + kQT, qs1, ds1, tx1, tz1, qs0, ds0, tx0, tz0);
  }
  // lane: key wk0 + 16kb + r, dims 16db + 4j + i; dka holds -dK / scale
  const size_t out_base = (size_t)chunk * ((size_t)grid.z * nkeys_total * HD);
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) {
    const int key = wk0 + 16 * kb + r;
    if (key >= nkeys_total) continue;
    const size_t off = out_base + ((size_t)bh * nkeys_total + key) * HD;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      store4(dk_out + off + 16 * db + 4 * j, dka[kb][db], -scale);
      store4(dv_out + off + 16 * db + 4 * j, dva[kb][db], 1.0f);
    }
  }
}


// The pass as its own launch.
template <int HD, int NW, bool BALL, bool MASK = true, bool PS = false, int KBW = 2>
__global__ void __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(PS && !MASK ? 3 : 1)))
dense_bwd_kv_dma_kernel(KvArgs a) {
  BSA_KV_LDS(L);
  kv_dma_body<HD, NW, BALL, MASK, PS, KBW>(L, gridDim, blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z),
                                          a);
}

// The compressed pass (prescaled keys, unmasked) and the ball pass (one 16-key block per
// wave) in one launch: the compressed workgroups first, then the ball workgroups, which
// fill the CUs that the compressed pass's last round leaves idle (its workgroups are long
// and few, about 2.7 per CU slot) and overlap their HBM traffic with its MFMA work.
template <int HD, bool BMASK>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3)))
dense_bwd_kv_pair_kernel(KvArgs cmp, dim3 cgrid, KvArgs ball, dim3 bgrid) {
  BSA_KV_LDS(L);
  const unsigned ncmp = cgrid.x * cgrid.y * cgrid.z;
  if (blockIdx.x < ncmp)
    kv_dma_body<HD, 4, false, false, true, 2>(L, cgrid, blockIdx.x, cmp);
  else
    kv_dma_body<HD, 4, true, BMASK, false, 1>(L, bgrid, blockIdx.x - ncmp, ball);
}

// ==== selection branch, query-major: dQ over the tokens of the selected blocks ====
template <typename T, int HD>
__global__ void __launch_bounds__(256) slc_bwd_q_kernel(const T* q, const T* k, const T* v, const T* dout,
                                                        const uint8_t* valid_all, const int* sel, QTerms qt, int H,
                                                        int N, int ls, int kk, int g, float sl2, float scale,
                                                        float* dq) {
  constexpr int NCH = HD / 32, DB = HD / 16;
  constexpr int VSTR = 32 + 4;
  typedef typename Chunk<T>::type CT;
  __shared__ __attribute__((aligned(16))) T kt_all[4][HD * VSTR];
  __shared__ int sub_all[4][kMaxSub];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15, j = lane >> 4;
  const int b = blockIdx.z, h = blockIdx.y;
  const long long bh = (long long)b * H + h;
  const int wq0 = (blockIdx.x * 4 + wid) * 16;
  const int G = g >= 16 ? 1 : 16 / g;
  const int p0 = wq0 / g;
  const int my_gi = g >= 16 ? 0 : r / g;
  const int ngroups = N / g;
  const T* kh = k + bh * N * HD;
  const T* vh = v + bh * N * HD;
  const uint8_t* val = valid_all ? valid_all + (size_t)b * N : nullptr;
  const int* selp = sel + ((size_t)bh * ngroups + p0) * kk;
  T* kt = kt_all[wid];
  int* sub = sub_all[wid];

  const int nsub = G * kk * (ls / 16);
  for (int e = lane; e < nsub; e += 64) {
    const int slot = (e * 16) / ls;
    const int gi = slot / kk;
    const int id = selp[gi * kk + slot % kk];
    sub[e] = id < 0 ? -1 : ((gi << 24) | (id * ls + (e * 16) % ls));
  }
  const long long row = bh * N + wq0 + r;
  CT qf[NCH], df[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    qf[c] = load_chunk(q + row * HD + 32 * c + 8 * j);
    df[c] = load_chunk(dout + row * HD + 32 * c + 8 * j);
  }
  const float4 tq = qt.t4[row];
  const float l2 = tq.x, gs = tq.y, dd = tq.z;
  f32x4 acc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  wave_sync();   // LDS regions are per wave
  vm_drain();

  for (int sb0 = 0; sb0 < nsub; sb0 += 2) {
    const int ent[2] = {sub[sb0], sb0 + 1 < nsub ? sub[sb0 + 1] : -1};
    CT kf[2][NCH], vf[2][NCH];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        kf[kb][c] = zero_chunk(kf[kb][c]);
        vf[kb][c] = zero_chunk(vf[kb][c]);
        if (ent[kb] >= 0) {
          const size_t o = (size_t)((ent[kb] & 0xFFFFFF) + r) * HD + 32 * c + 8 * j;
          kf[kb][c] = load_chunk(kh + o);
          vf[kb][c] = load_chunk(vh + o);
        }
      }
    bool ok[2][4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = ent[kb];
        ok[kb][i] = e >= 0 && (e >> 24) == my_gi && (val == nullptr || val[(e & 0xFFFFFF) + 4 * j + i]);
      }
    wave_sync();   // LDS regions are per wave
    for (int e = lane; e < 8 * (HD / 8); e += 64) {
      const int kq = e / (HD / 8), dc = (e % (HD / 8)) * 8;
      const int en = ent[kq >> 2];
      const T* rows[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) rows[u] = en >= 0 ? kh + (size_t)((en & 0xFFFFFF) + 4 * (kq & 3) + u) * HD : nullptr;
      stage_vt(rows, dc, kt, VSTR, 4 * kq);
    }
    wave_sync();   // LDS regions are per wave
    f32x4 s[2], dp[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
      dp[kb] = s[kb];
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        s[kb] = mma(kf[kb][c], qf[c], s[kb]);
        dp[kb] = mma(vf[kb][c], df[c], dp[kb]);
      }
    }
    float w8[8];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = ok[kb][i] ? fast_exp2(__builtin_fmaf(s[kb][i], sl2, -l2)) : 0.f;
        w8[4 * kb + i] = p * (dp[kb][i] - dd);
      }
    const CT dsf = make_chunk<T>(w8);
#pragma unroll
    for (int db = 0; db < DB; ++db) acc[db] = mma(load_4x2(&kt[(16 * db + r) * VSTR + 4 * j]), dsf, acc[db]);
  }
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    float* dst = dq + row * HD + 16 * db + 4 * j;
    float4 old = *reinterpret_cast<float4*>(dst);
    f32x4 val = acc[db] * scale;
    val[0] += old.x; val[1] += old.y; val[2] += old.z; val[3] += old.w;
    store4(dst, val, 1.0f);
  }
}

// ==== selection branch, key-major: dK, dV of each selection block from its groups ====
// (b,h,block) -> sorted list of the groups that selected it: pairs[seg_start .. seg_end).

// 16x16 MFMA with a 16-deep contraction: 4 values per lane group (k = 4*(L/16) + i).
// A comes as 4 raw storage elements (8 bytes bf16 / 16 bytes f32), B as 4 f32 values.
typedef short s16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ f32x4 mma16(const bf16_t* a, const float (&bv)[4], f32x4 c) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  const uint2 ar = *reinterpret_cast<const uint2*>(a);
  bf16x4 y = {(__bf16)bv[0], (__bf16)bv[1], (__bf16)bv[2], (__bf16)bv[3]};
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, ar), __builtin_bit_cast(s16x4, y), c, 0,
                                                   0, 0);
}
__device__ __forceinline__ f32x4 mma16(uint2 ar, const float (&bv)[4], f32x4 c) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  bf16x4 y = {(__bf16)bv[0], (__bf16)bv[1], (__bf16)bv[2], (__bf16)bv[3]};
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, ar), __builtin_bit_cast(s16x4, y), c, 0,
                                                   0, 0);
}
__device__ __forceinline__ f32x4 mma16(const float* a, const float (&bv)[4], f32x4 c) {
  const float4 ar = *reinterpret_cast<const float4*>(a);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(ar.x, bv[0], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(ar.y, bv[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(ar.z, bv[2], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(ar.w, bv[3], c, 0, 0, 0);
  return c;
}

__global__ void slc_pairs_kernel(const int* sel, long long total, int kk, int ngroups, int nblk, uint32_t sentinel,
                                 uint32_t* keys, uint32_t* vals) {
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const long long row = i / kk;             // (bh, p)
  const int p = (int)(row % ngroups);
  const long long bh = row / ngroups;
  const int id = sel[i];
  keys[i] = id < 0 ? sentinel : (uint32_t)(bh * nblk + id);
  vals[i] = (uint32_t)p;
}

__global__ void fill_kernel(int* x, long long n, int v) {
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) x[i] = v;
}

__global__ void seg_bounds_kernel(const uint32_t* keys, long long total, uint32_t sentinel, int* seg_start,
                                  int* seg_end) {
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const uint32_t kx = keys[i];
  if (kx == sentinel) return;
  if (i == 0 || keys[i - 1] != kx) seg_start[kx] = (int)i;
  if (i == total - 1 || keys[i + 1] != kx) seg_end[kx] = (int)(i + 1);
}

// bf16 variant of the selection query-major pass: each wave double-buffers its key tiles
// (the 32 K rows and 32 V rows of two sub-blocks) in LDS, filled by direct global->LDS loads
// one tile ahead (two distinct LDS objects, straight-line body unrolled by two; tiles past
// the end are loaded from row 0 and masked). K^T for the dQ product comes from transpose
// reads of the K tile. Key validity is gathered into 16-bit masks with the sub-block list.
template <int HD, int NW>
__global__ void __launch_bounds__(NW * 64) slc_bwd_q_dma_kernel(const bf16_t* q, const bf16_t* k, const bf16_t* v,
                                                                const bf16_t* dout, const uint8_t* valid_all,
                                                                const int* sel, QTerms qt, int H, int N, int ls,
                                                                int kk, int g, float sl2, float scale, float* dq) {
  constexpr int NCH = HD / 32, DB = HD / 16;
  constexpr int TILE = 32 * HD;    // one 32-key tile
  constexpr int SLOT = 2 * TILE;   // K tile, V tile
  typedef bf16x8 CT;
  __shared__ __attribute__((aligned(16))) bf16_t buf0[NW * SLOT], buf1[NW * SLOT];
  __shared__ int sub_all[NW][kMaxSub];
  __shared__ uint32_t okm_all[NW][kMaxSub];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15, j = lane >> 4;
  const dim3 blk = xcd_grouped_block((int)gridDim.x);   // one head's groups per XCD run
  const int b = blk.z, h = blk.y;
  const long long bh = (long long)b * H + h;
  const int wq0 = (blk.x * NW + wid) * 16;
  const int G = g >= 16 ? 1 : 16 / g;
  const int p0 = wq0 / g;
  const int my_gi = g >= 16 ? 0 : r / g;
  const int ngroups = N / g;
  const bf16_t* kh = k + bh * N * HD;
  const bf16_t* vh = v + bh * N * HD;
  const uint8_t* val = valid_all ? valid_all + (size_t)b * N : nullptr;
  const int* selp = sel + ((size_t)bh * ngroups + p0) * kk;
  int* sub = sub_all[wid];
  uint32_t* okm = okm_all[wid];

  const int nsub = G * kk * (ls / 16);
  for (int e = lane; e < nsub; e += 64) {
    const int slot = (e * 16) / ls;
    const int gi = slot / kk;
    const int id = selp[gi * kk + slot % kk];
    const int tok0 = id * ls + (e * 16) % ls;
    sub[e] = id < 0 ? -1 : ((gi << 24) | tok0);
    uint32_t m = 0;
    if (id >= 0) {
      m = 0xFFFFu;
      if (val)
        for (int t = 0; t < 16; ++t)
          if (!val[tok0 + t]) m &= ~(1u << t);
    }
    okm[e] = m;
  }
  const long long row = bh * N + wq0 + r;
  CT qf[NCH], df[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    qf[c] = load_chunk(q + row * HD + 32 * c + 8 * j);
    df[c] = load_chunk(dout + row * HD + 32 * c + 8 * j);
  }
  const float4 tr = qt.t4[row];   // log2 LSE - log2 s, s, R of this lane's query
  const float l2 = tr.x, gs = tr.y, dd = tr.z;
  f32x4 acc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  vm_drain();
  wave_sync();   // LDS regions are per wave

  const int nt = __builtin_amdgcn_readfirstlane((nsub + 1) / 2);   // 32-key tiles
  auto issue = [&](int t, bf16_t* slot) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int e = 2 * t + kb < nsub ? sub[2 * t + kb] : -1;
      const int r0 = e >= 0 ? (e & 0xFFFFFF) : 0;
      bf16_t* base = slot + wid * SLOT + kb * 16 * HD;
      dma_tile_full<HD, 16, 1>(base, kh + (size_t)r0 * HD, 0, lane);
      dma_tile_full<HD, 16, 1>(base + TILE, vh + (size_t)r0 * HD, 0, lane);
    }
  };
  auto step = [&](int t, const bf16_t* cur, bf16_t* next) {
    vm_drain();   // this tile has landed
    issue(t + 1, next);
    const bf16_t* kt = cur + wid * SLOT;
    const bf16_t* vt = kt + TILE;
    uint32_t m[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int se = 2 * t + kb;
      const int e = t < nt && se < nsub ? sub[se] : -1;
      m[kb] = e >= 0 && (e >> 24) == my_gi ? okm[se] : 0u;
    }
    // dp starts from -dd, so the product yields dP - dd directly
    f32x4 sv[2], dp[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      sv[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
      dp[kb] = f32x4{-dd, -dd, -dd, -dd};
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        sv[kb] = mma(lds_row_chunk<HD>(kt, 16 * kb + r, 4 * c + j), qf[c], sv[kb]);
        dp[kb] = mma(lds_row_chunk<HD>(vt, 16 * kb + r, 4 * c + j), df[c], dp[kb]);
      }
    }
    float w8[8];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) w8[4 * kb + i] = fast_exp2(__builtin_fmaf(sv[kb][i], sl2, -l2)) * dp[kb][i];
    // keys that are padding, of another lane's group or of a missing block contribute 0 (the
    // loaded rows are finite); skipped when every key of the tile is seen by every lane
    if (__builtin_amdgcn_ballot_w64((m[0] & m[1]) != 0xFFFFu) != 0) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (!((m[kb] >> (4 * j + i)) & 1u)) w8[4 * kb + i] = 0.f;
    }
    const CT dsf = make_chunk<bf16_t>(w8);
#pragma unroll
    for (int db = 0; db < DB; ++db) acc[db] = mma(lds_tr_chunk_nowait<HD>(kt, 0, 16 * db, lane), dsf, acc[db]);
  };
  issue(0, buf0);
  for (int t = 0; t < nt; t += 2) {   // straight-line body
    step(t, buf0, buf1);
    step(t + 1, buf1, buf0);
  }
  vm_drain();   // the loads past the end have landed
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    float* dst = dq + row * HD + 16 * db + 4 * j;
    float4 old = *reinterpret_cast<float4*>(dst);
    f32x4 val4 = acc[db] * scale;
    val4[0] += old.x; val4[1] += old.y; val4[2] += old.z; val4[3] += old.w;
    store4(dst, val4, 1.0f);
  }
}

// One workgroup per (b, h, block): wave w takes the block's groups w, w+4, ... (prefetching
// the next group's rows while computing the current one) and keeps partial dK, dV in
// registers; the four partials are then summed in wave order through LDS.
template <typename T, int HD, int KBW>
__global__ void __launch_bounds__(256) slc_bwd_kv_kernel(const T* q, const T* k, const T* v, const T* dout,
                                                         const uint8_t* valid_all, const uint32_t* groups,
                                                         const int* seg_start, const int* seg_end, QTerms qt, int H,
                                                         int N, int ls, int g, long long nseg, float sl2, float scale,
                                                         float* dk, float* dv) {
  constexpr int NCH = HD / 32, DB = HD / 16;
  constexpr int TSTR = 16 + 4;
  typedef typename Chunk<T>::type CT;
  __shared__ __attribute__((aligned(16))) T qtr_all[4][HD * TSTR];
  __shared__ __attribute__((aligned(16))) T dtr_all[4][HD * TSTR];
  __shared__ __attribute__((aligned(16))) float red[2][KBW * 16 * HD];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15, j = lane >> 4;
  const long long seg = blockIdx.x;
  const int nblk = N / ls;
  const long long bh = seg / nblk;
  const int blk = (int)(seg % nblk);
  const int b = (int)(bh / H);
  const int s0 = seg_start[seg], s1 = seg_end[seg];
  if (s1 <= s0) return;                     // uniform over the workgroup
  T* qtr = qtr_all[wid];
  T* dtr = dtr_all[wid];
  const T* qh = q + (size_t)bh * N * HD;
  const T* dh = dout + (size_t)bh * N * HD;
  const uint8_t* val = valid_all ? valid_all + (size_t)b * N : nullptr;

  CT kf[KBW][NCH], vf[KBW][NCH];
  bool kok[KBW];
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) {
    const int key = blk * ls + 16 * kb + r;
    kok[kb] = val == nullptr || val[key];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      kf[kb][c] = load_chunk(k + ((size_t)bh * N + key) * HD + 32 * c + 8 * j);
      vf[kb][c] = load_chunk(v + ((size_t)bh * N + key) * HD + 32 * c + 8 * j);
    }
  }
  f32x4 dka[KBW][DB], dva[KBW][DB];
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb)
#pragma unroll
    for (int db = 0; db < DB; ++db) { dka[kb][db] = f32x4{0.f, 0.f, 0.f, 0.f}; dva[kb][db] = dka[kb][db]; }

  const int qblocks = g >= 16 ? g / 16 : 1;
  const int qrows = g >= 16 ? 16 : g;       // real rows of each 16-query block
  const int nwork = (s1 - s0) * qblocks;    // (group, 16-query block) items of this block
  // per-item inputs: A rows of Q and dO (lane row = query r) and the terms of rows 4j+i
  CT aq[NCH], ad[NCH];
  float lv[4], dvv[4], gv[4];
  auto fetch = [&](int item) {
    const int e = s0 + item / qblocks;
    const int qr0 = (int)groups[e] * g + 16 * (item % qblocks);
    const bool rok = r < qrows;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      aq[c] = zero_chunk(aq[c]);
      ad[c] = zero_chunk(ad[c]);
      if (rok) {
        aq[c] = load_chunk(qh + (size_t)(qr0 + r) * HD + 32 * c + 8 * j);
        ad[c] = load_chunk(dh + (size_t)(qr0 + r) * HD + 32 * c + 8 * j);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rr = 4 * j + i;
      lv[i] = __builtin_huge_valf();
      dvv[i] = 0.f;
      gv[i] = 0.f;
      if (rr < qrows) {
        const long long row = bh * N + qr0 + rr;
        const float4 t = qt.t4[row];
        lv[i] = t.x;
        gv[i] = t.y;
        dvv[i] = t.z;
      }
    }
  };
  if (wid < nwork) fetch(wid);
  vm_drain();
  for (int item = wid; item < nwork; item += 4) {
    CT cq[NCH], cd[NCH];
    float cl[4], cdv[4], cg[4];
#pragma unroll
    for (int c = 0; c < NCH; ++c) { cq[c] = aq[c]; cd[c] = ad[c]; }
#pragma unroll
    for (int i = 0; i < 4; ++i) { cl[i] = lv[i]; cdv[i] = dvv[i]; cg[i] = gv[i]; }
    if (item + 4 < nwork) fetch(item + 4);   // next item in flight
    // Q^T and dO^T of the 16 queries, written from the row fragments this lane holds
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        qtr[(32 * c + 8 * j + e) * TSTR + r] = chunk_elem(cq[c], e);
        dtr[(32 * c + 8 * j + e) * TSTR + r] = chunk_elem(cd[c], e);
      }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int kb = 0; kb < KBW; ++kb) {
      f32x4 sv = f32x4{0.f, 0.f, 0.f, 0.f}, dp = sv;
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        sv = mma(cq[c], kf[kb][c], sv);
        dp = mma(cd[c], vf[kb][c], dp);
      }
      float pg[4], dsv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float pr = kok[kb] ? fast_exp2(__builtin_fmaf(sv[i], sl2, -cl[i])) : 0.f;
        pg[i] = pr;
        dsv[i] = pr * (dp[i] - cdv[i]);
      }
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        dva[kb][db] = mma16(&dtr[(16 * db + r) * TSTR + 4 * j], pg, dva[kb][db]);
        dka[kb][db] = mma16(&qtr[(16 * db + r) * TSTR + 4 * j], dsv, dka[kb][db]);
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  // fixed-order sum of the four waves' partials: wave 0 accumulates waves 1, 2, 3
  for (int w = 1; w < 4; ++w) {
    __syncthreads();
    if (wid == w) {
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb)
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const int o = (16 * kb + r) * HD + 16 * db + 4 * j;
          *reinterpret_cast<f32x4*>(&red[0][o]) = dka[kb][db];
          *reinterpret_cast<f32x4*>(&red[1][o]) = dva[kb][db];
        }
    }
    __syncthreads();
    if (wid == 0) {
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb)
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const int o = (16 * kb + r) * HD + 16 * db + 4 * j;
          dka[kb][db] += *reinterpret_cast<const f32x4*>(&red[0][o]);
          dva[kb][db] += *reinterpret_cast<const f32x4*>(&red[1][o]);
        }
    }
  }
  if (wid != 0) return;
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) {
    const size_t off = ((size_t)bh * N + blk * ls + 16 * kb + r) * HD;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      float* pk = dk + off + 16 * db + 4 * j;
      float* pv = dv + off + 16 * db + 4 * j;
      float4 ok4 = *reinterpret_cast<float4*>(pk), ov4 = *reinterpret_cast<float4*>(pv);
      f32x4 a = dka[kb][db] * scale, c = dva[kb][db];
      a[0] += ok4.x; a[1] += ok4.y; a[2] += ok4.z; a[3] += ok4.w;
      c[0] += ov4.x; c[1] += ov4.y; c[2] += ov4.z; c[3] += ov4.w;
      store4(pk, a, 1.0f);
      store4(pv, c, 1.0f);
    }
  }
}

constexpr int kCmpChunks = 8;   // query chunks of the compressed branch's key-major pass

// Query-major pass launcher: bf16 layers take the direct-load kernel, f32 layers the
// register-staged one. Non-ball (compressed) launches of bf16 layers read prescaled keys.
template <typename T, int HD, int QB, bool BALL, bool ADD>
void launch_bwd_q(dim3 grid, hipStream_t st, const T* q, const T* k, const T* v, const T* dout,
                  const uint8_t* kvalid, QTerms qt, int H, int N, int nkeys_total, int m, float sl2, float scale,
                  float* dq) {
  if constexpr (sizeof(T) == 2) {
    if (kvalid == nullptr && (BALL ? m : nkeys_total) % kKT == 0)
      hipLaunchKernelGGL((dense_bwd_q_dma_kernel<HD, QB, BALL, ADD, false, !BALL>), grid, dim3(256), 0, st, q, k, v,
                         dout, kvalid, qt, H, N, nkeys_total, m, sl2, scale, dq);
    else
      hipLaunchKernelGGL((dense_bwd_q_dma_kernel<HD, QB, BALL, ADD, true, !BALL>), grid, dim3(256), 0, st, q, k, v,
                         dout, kvalid, qt, H, N, nkeys_total, m, sl2, scale, dq);
  }
  else
    hipLaunchKernelGGL((dense_bwd_q_kernel<T, HD, QB, BALL, ADD>), grid, dim3(256), 0, st, q, k, v, dout, kvalid, qt,
                       H, N, nkeys_total, m, sl2, scale, dq);
}

// Key-major pass launcher: bf16 layers take the direct-load kernel, f32 layers the
// register-staged one. Non-ball (compressed) launches of bf16 layers read prescaled keys.
template <typename T, int HD, int NW, bool BALL, int KBW = 2>
void launch_bwd_kv(dim3 grid, hipStream_t st, const T* q, const T* k, const T* v, const T* dout,
                   const uint8_t* kvalid, QTerms qt, int H, int N, int nkeys_total, int m, int nchunks, float sl2,
                   float scale, float* dk, float* dv) {
  if constexpr (sizeof(T) == 2) {
    const KvArgs a{q, k, v, dout, kvalid, qt, H, N, nkeys_total, m, nchunks, sl2, scale, dk, dv};
    if (kvalid == nullptr && nkeys_total % (NW * 16 * KBW) == 0)
      hipLaunchKernelGGL((dense_bwd_kv_dma_kernel<HD, NW, BALL, false, !BALL, KBW>), grid, dim3(NW * 64), 0, st, a);
    else
      hipLaunchKernelGGL((dense_bwd_kv_dma_kernel<HD, NW, BALL, true, !BALL, KBW>), grid, dim3(NW * 64), 0, st, a);
  }
  else
    hipLaunchKernelGGL((dense_bwd_kv_kernel<T, HD, NW, BALL>), grid, dim3(NW * 64), 0, st, q, k, v, dout, kvalid, qt,
                       H, N, nkeys_total, m, nchunks, sl2, scale, dk, dv);
}

// The backward pass in stages; bsa_backward orders them across its two streams (the
// stages' buffer dependencies are listed with BwdStage in kernels.hpp).
template <typename T, int HD>
hipError_t bwd_stage_impl(const Dims& D, const BwdArgs& A, BwdStage stage, hipStream_t st) {
  const long long rows = D.rows();
  const float sl2 = D.scale * kLog2e;
  const int nct = D.N / D.l;
  // compressed tokens (and the coarse queries of Eq. 15) in the storage type, as the
  // forward pass consumed them (cast in the prep stage)
  const T* kc = D.bf16 ? (const T*)A.kc_lp : (const T*)A.kcmp;
  const T* vc = D.bf16 ? (const T*)A.vc_lp : (const T*)A.vcmp;
  const T* qcl = D.bf16 ? (const T*)A.qc_lp : (const T*)A.qcmp;
  const float4* t4 = (const float4*)A.terms;
  QTerms qball{t4};
  QTerms qcmp{t4 + rows};
  QTerms qslc{t4 + 2 * rows};
  QTerms qcoarse{(const float4*)A.t4c};
  const T* q = (const T*)A.q;
  const T* k = (const T*)A.k;
  const T* v = (const T*)A.v;
  const T* dout = (const T*)A.dout;
  const T* docl = (const T*)A.doc;
  switch (stage) {
    case BwdStage::prep: {
      if (D.bf16) {
        const long long n = D.cmp_rows() * HD;
        // the compressed keys carry the softmax scale times log2(e), as in the forward
        hipLaunchKernelGGL(cast_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, A.kcmp, n,
                           cmp_key_scale(D), (T*)A.kc_lp);
        hipLaunchKernelGGL(cast_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, A.vcmp, n, 1.0f,
                           (T*)A.vc_lp);
        if (D.gcmp)
          hipLaunchKernelGGL(cast_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, A.qcmp, n, 1.0f,
                             (T*)A.qc_lp);
      }
      // store_lse = 0: each branch's log-sum-exp rows are recomputed by its forward kernel
      // without the value products (the same tiles and order, so they equal the stored ones)
      const float* lse = A.lse;
      if (!D.store_lse) {
        hipError_t e = hipSuccess;
        BSA_PHASE("bwd.lse", st, {
          e = launch_ball_fwd(D, A.q, A.k, A.v, A.valid, nullptr, A.lse_ws, st);
          if (e == hipSuccess && D.gcmp) {
            e = launch_cmp_coarse_fwd(D, qcl, kc, vc, A.valid ? A.cvalid : nullptr, nullptr, A.lsec_ws, st);
            if (e == hipSuccess)
              e = launch_expand_coarse(D, nullptr, A.lsec_ws, A.valid, nullptr, A.lse_ws + rows, st);
          } else if (e == hipSuccess) {
            e = launch_cmp_fwd(D, A.q, kc, vc, A.valid, A.valid ? A.cvalid : nullptr, nullptr, A.lse_ws + rows, st);
          }
          if (e == hipSuccess)
            e = D.g == 1 ? launch_slc1_fwd(D, A.q, A.k, A.v, A.valid, A.sel, A.s1, nullptr, A.lse_ws + 2 * rows, st)
                         : launch_slc_fwd(D, A.q, A.k, A.v, A.valid, A.sel, nullptr, A.lse_ws + 2 * rows, st);
        });
        if (e != hipSuccess) return e;
        lse = A.lse_ws;
      }
      // per-branch row sums, the packed row terms and the gate gradient
      BSA_PHASE("bwd.gate", st, {
        hipLaunchKernelGGL(gate_bwd_rows_kernel<T>, dim3((unsigned)((rows * 8 + 255) / 256)), dim3(256), 0, st,
                           dout, (const T*)A.o_branch, A.o_cmp, rows, HD, lse, A.gate, D.H, D.N, A.R,
                           (float4*)A.terms);
        hipLaunchKernelGGL(gate_bwd_kernel, dim3((D.B * D.N + 255) / 256), dim3(256), 0, st, A.R, A.gate, A.valid,
                           D.B, D.H, D.N, A.dgate);
      });
      // group compression: the coarse queries' dO and row terms
      if (D.gcmp) {
        const long long n = D.cmp_rows() * HD;
        hipLaunchKernelGGL(coarse_rows_bwd_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, dout,
                           t4 + rows, A.ocmp, A.valid, D.H, D.N, D.l, HD, D.cmp_rows(), (T*)A.doc, (float4*)A.t4c);
      }
      break;
    }
    case BwdStage::kv_ball:   // dK, dV of the ball branch (written)
      BSA_PHASE("bwd.kv_ball", st, {
        // bf16: one 16-key block per wave (64 keys per workgroup; ball_size >= 64): half the
        // registers, twice the waves for this HBM-bound pass
        if constexpr (sizeof(T) == 2) {
          (launch_bwd_kv<T, HD, 4, true, 1>)(dim3(D.N / 64, 1, D.B * D.H), st, q, k, v, dout, A.valid, qball, D.H,
                                           D.N, D.N, D.m, 1, sl2, D.scale, A.dk, A.dv);
        } else if (D.m >= 128) {
          (launch_bwd_kv<T, HD, 4, true>)(dim3(D.N / 128, 1, D.B * D.H), st, q, k, v, dout, A.valid, qball, D.H,
                                        D.N, D.N, D.m, 1, sl2, D.scale, A.dk, A.dv);
        } else {
          (launch_bwd_kv<T, HD, 2, true>)(dim3(D.N / 64, 1, D.B * D.H), st, q, k, v, dout, A.valid, qball, D.H,
                                        D.N, D.N, D.m, 1, sl2, D.scale, A.dk, A.dv);
        }
      });
      break;
    case BwdStage::kv_pair: {   // kv_ball and kv_cmp, in one launch where both are unmasked bf16 passes
      if constexpr (sizeof(T) == 2) {
        const int nq = D.gcmp ? nct : D.N;
        const int nch = nq / kCmpChunks >= kQT ? kCmpChunks : 1;
        const dim3 cg((nct + 127) / 128, nch, D.B * D.H), bg(D.N / 64, 1, D.B * D.H);
        if (A.valid == nullptr && nct % 128 == 0 && D.N % 64 == 0 && D.m % 64 == 0 && (cg.x * cg.y * cg.z) % 8 == 0) {
          const KvArgs cmp{D.gcmp ? qcl : q, kc, vc, D.gcmp ? docl : dout, nullptr, D.gcmp ? qcoarse : qcmp, D.H, nq,
                           nct, D.m, nch, sl2, D.scale, A.dkc_part, A.dvc_part};
          const KvArgs ball{q, k, v, dout, nullptr, qball, D.H, D.N, D.N, D.m, 1, sl2, D.scale, A.dk, A.dv};
          BSA_PHASE("bwd.kv", st,
                    hipLaunchKernelGGL((dense_bwd_kv_pair_kernel<HD, false>),
                                       dim3(cg.x * cg.y * cg.z + bg.x * bg.y * bg.z), dim3(256), 0, st, cmp, cg, ball,
                                       bg));
          const long long n = D.cmp_rows() * HD;
          hipLaunchKernelGGL(sum_chunks_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, A.dkc_part, nch,
                             n, A.dkc);
          hipLaunchKernelGGL(sum_chunks_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, A.dvc_part, nch,
                             n, A.dvc);
          break;
        }
      }
      hipError_t e = bwd_stage_impl<T, HD>(D, A, BwdStage::kv_ball, st);
      if (e != hipSuccess) return e;
      return bwd_stage_impl<T, HD>(D, A, BwdStage::kv_cmp, st);
    }
    case BwdStage::kv_cmp: {   // dK^, dV^ of the compressed branch: chunked partials, fixed-order sum
      const int nq = D.gcmp ? nct : D.N;   // query rows: tokens, or coarse queries (Eq. 15)
      const int nch = nq / kCmpChunks >= kQT ? kCmpChunks : 1;
      BSA_PHASE("bwd.kv_cmp", st,
      (launch_bwd_kv<T, HD, 4, false>)(dim3((nct + 127) / 128, nch, D.B * D.H), st, D.gcmp ? qcl : q, kc, vc,
                                     D.gcmp ? docl : dout, A.valid ? A.cvalid : nullptr, D.gcmp ? qcoarse : qcmp,
                                     D.H, nq, nct, D.m, nch, sl2, D.scale, A.dkc_part, A.dvc_part));
      const long long n = D.cmp_rows() * HD;
      hipLaunchKernelGGL(sum_chunks_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, A.dkc_part, nch, n,
                         A.dkc);
      hipLaunchKernelGGL(sum_chunks_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, A.dvc_part, nch, n,
                         A.dvc);
      break;
    }
    case BwdStage::dq_ball:   // dQ of the ball branch (written)
      BSA_PHASE("bwd.dq_ball", st, {
        if (D.m >= 128)
          (launch_bwd_q<T, HD, 2, true, false>)(dim3(D.N / 128, D.H, D.B), st, q, k, v, dout, A.valid, qball, D.H,
                                                D.N, D.N, D.m, sl2, D.scale, A.dq);
        else
          (launch_bwd_q<T, HD, 1, true, false>)(dim3(D.N / 64, D.H, D.B), st, q, k, v, dout, A.valid, qball, D.H,
                                                D.N, D.N, D.m, sl2, D.scale, A.dq);
      });
      break;
    case BwdStage::dq_cmp:   // dQ of the compressed branch (added), or the coarse queries' (written)
      BSA_PHASE("bwd.dq_cmp", st, {
        if (!D.gcmp && D.N % 128 == 0)
          (launch_bwd_q<T, HD, 2, false, true>)(dim3(D.N / 128, D.H, D.B), st, q, kc, vc, dout,
                                                A.valid ? A.cvalid : nullptr, qcmp, D.H, D.N, nct, D.m, sl2, D.scale,
                                                A.dq);
        else if (!D.gcmp)   // 64 token slots
          (launch_bwd_q<T, HD, 1, false, true>)(dim3(D.N / 64, D.H, D.B), st, q, kc, vc, dout,
                                                A.valid ? A.cvalid : nullptr, qcmp, D.H, D.N, nct, D.m, sl2, D.scale,
                                                A.dq);
        else if (nct % 128 == 0)
          (launch_bwd_q<T, HD, 2, false, false>)(dim3(nct / 128, D.H, D.B), st, qcl, kc, vc, docl,
                                                 A.valid ? A.cvalid : nullptr, qcoarse, D.H, nct, nct, D.m, sl2,
                                                 D.scale, A.dqc);
        else
          (launch_bwd_q<T, HD, 1, false, false>)(dim3(nct / 64, D.H, D.B), st, qcl, kc, vc, docl,
                                                 A.valid ? A.cvalid : nullptr, qcoarse, D.H, nct, nct, D.m, sl2,
                                                 D.scale, A.dqc);
      });
      break;
    case BwdStage::dq_slc:   // dQ of the selection branch (added); groups of g >= 8 only
      BSA_PHASE("bwd.dq_slc", st, {
        if constexpr (sizeof(T) == 2) {
          constexpr int NW = 2;
          hipLaunchKernelGGL((slc_bwd_q_dma_kernel<HD, NW>), dim3(D.N / (16 * NW), D.H, D.B), dim3(64 * NW), 0, st,
                             q, k, v, dout, A.valid, A.sel, qslc, D.H, D.N, D.ls, D.k, D.g, sl2, D.scale, A.dq);
        } else {
          hipLaunchKernelGGL((slc_bwd_q_kernel<T, HD>), dim3(D.N / 64, D.H, D.B), dim3(256), 0, st, q, k, v, dout,
                             A.valid, A.sel, qslc, D.H, D.N, D.ls, D.k, D.g, sl2, D.scale, A.dq);
        }
      });
      break;
  }
  return hipGetLastError();
}

// bf16 variant of the selection key-major pass. NWV waves share a block's items. Blocks
// with at most kSlcLightItems items take one wave per workgroup: it walks all of the
// block's items, which spreads the start-up latency of the K/V fragments, the row list and
// the first item over more items, and a workgroup of one wave needs only 15 KB of LDS, so
// eight blocks run per CU. Blocks chosen by many groups (selection can concentrate on a
// few blocks) take a second launch of persistent workgroups of eight waves (four where a
// wave holds four key blocks), so that no single wave walks a long list; each launch
// skips the other's blocks. Each wave keeps a ring of three item
// slots in LDS (16 query rows of Q and dO and their packed row terms), filled by direct
// global->LDS loads two items ahead. The slots are three distinct LDS objects and the item
// loop is unrolled by three with a straight-line body (steps past the end of the list
// compute with zero weights), so reads of a slot wait only for that slot's loads. Item row
// indices come from a per-wave list in LDS. The dK^T and dV^T products take their Q^T and
// dO^T operands from transpose reads of the slot tiles.
template <int HD, int KBW, int NWV>
__global__ void __launch_bounds__(64 * NWV) slc_bwd_kv_dma_kernel(const bf16_t* q, const bf16_t* k, const bf16_t* v,
                                                             const bf16_t* dout, const uint8_t* valid_all,
                                                             const uint32_t* groups, const int* seg_start,
                                                             const int* seg_end, QTerms qt, int H, int N, int ls,
                                                             int g, long long nseg, float sl2, float scale, float* dk,
                                                             float* dv, int min_items, int max_items) {
  constexpr int NCH = HD / 32, DB = HD / 16;
  constexpr int SL = 16 * HD;             // elements of one 16-row tile
  constexpr int SLOT = 2 * SL + 64 * 8;   // one wave's slot: Q tile, dO tile, 64 lanes' row terms
  constexpr int kRound = 128;             // items per wave per round of the row list
  typedef bf16x8 CT;
  __shared__ __attribute__((aligned(16))) bf16_t ring0[NWV * SLOT], ring1[NWV * SLOT], ring2[NWV * SLOT];
  __shared__ int rows_all[NWV][kRound];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int r = lane & 15, j = lane >> 4;
  // one block of the selection: its partial dK/dV over its items, added into dk/dv
  auto block = [&](long long seg) {
    const int nblk = N / ls;
    const long long bh = seg / nblk;
    const int blk = (int)(seg % nblk);
    const int b = (int)(bh / H);
    const int s0 = seg_start[seg], s1 = seg_end[seg];
    if (s1 <= s0) return;                     // uniform over the workgroup
    const bf16_t* qh = q + (size_t)bh * N * HD;
    const bf16_t* dh = dout + (size_t)bh * N * HD;
    const float4* th = qt.t4 + (size_t)bh * N;
    const uint8_t* val = valid_all ? valid_all + (size_t)b * N : nullptr;
    int* rows = rows_all[wid];

    const int qblocks = g >= 16 ? g / 16 : 1;
    const int qrows = g >= 16 ? 16 : g;       // real rows of each 16-query block
    const int nwork = (s1 - s0) * qblocks;    // (group, 16-query block) items of this block
    if (nwork < min_items || nwork > max_items) return;   // the other launch's block
    const int nmine = nwork > wid ? (nwork - wid + NWV - 1) / NWV : 0;   // items w, w+NWV, ... of this wave

    CT kf[KBW][NCH], vf[KBW][NCH];
    bool kok[KBW];
  #pragma unroll
    for (int kb = 0; kb < KBW; ++kb) {
      const int key = blk * ls + 16 * kb + r;
      kok[kb] = val == nullptr || val[key];
  #pragma unroll
      for (int c = 0; c < NCH; ++c) {
        kf[kb][c] = load_chunk(k + ((size_t)bh * N + key) * HD + 32 * c + 8 * j);
        vf[kb][c] = load_chunk(v + ((size_t)bh * N + key) * HD + 32 * c + 8 * j);
      }
    }
    f32x4 dka[KBW][DB], dva[KBW][DB];
  #pragma unroll
    for (int kb = 0; kb < KBW; ++kb)
  #pragma unroll
      for (int db = 0; db < DB; ++db) { dka[kb][db] = f32x4{0.f, 0.f, 0.f, 0.f}; dva[kb][db] = dka[kb][db]; }

    int cnt = 0;   // items of the current round
    // item i's rows into a slot (past the round: a repeat of the last item, never used);
    // every lane loads a row term (lanes 16-63 repeat rows 0-15), so no load sits under a
    // lane mask
    auto issue = [&](int i, bf16_t* slot) {
      const int qr0 = rows[min(i, cnt - 1)];
      bf16_t* base = slot + wid * SLOT;
      // an item's 16 rows start at group * g: for g < 16 the last group's tile reaches g rows
      // past the end (rows clamp; those rows have zero weight)
      dma_tile<HD, 16, 1>(base, qh, qr0, N, 0, lane);
      dma_tile<HD, 16, 1>(base + SL, dh, qr0, N, 0, lane);
      __builtin_amdgcn_global_load_lds(th + min(qr0 + (lane & 15), N - 1), base + 2 * SL, 16, 0, 0);
    };
    // global->LDS loads per item: waiting until at most this many are outstanding leaves
    // only the next item's in flight
    constexpr int kPerItem = 2 * (HD / 32) + 1;
    auto step = [&](int i, const bf16_t* cur, bf16_t* next) {
      __builtin_amdgcn_s_waitcnt(0x0F70 | kPerItem);   // vmcnt(kPerItem): this slot has landed
      issue(i + 2, next);
      const bf16_t* qs = cur + wid * SLOT;
      const bf16_t* ds = qs + SL;
      const float4* ts = reinterpret_cast<const float4*>(qs + 2 * SL);
      const bool live = i < cnt;   // steps past the end of the round compute with zero weights
      CT aq[NCH], ad[NCH];
  #pragma unroll
      for (int c = 0; c < NCH; ++c) {
        aq[c] = lds_row_chunk<HD>(qs, r, 4 * c + j);
        ad[c] = lds_row_chunk<HD>(ds, r, 4 * c + j);
      }
      float cl[4], cg[4], cdv[4];
  #pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        const float4 t = ts[4 * j + ii];                  // log2 LSE - log2 s, s, R
        cl[ii] = live && 4 * j + ii < qrows ? t.x : __builtin_huge_valf();
        cg[ii] = t.y;
        cdv[ii] = t.z;
      }
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
        for (int ii = 0; ii < 4; ++ii) {
          const float pr = kok[kb] ? fast_exp2(__builtin_fmaf(sv[ii], sl2, -cl[ii])) : 0.f;
          pg[ii] = pr;
          dsv[ii] = pr * (dp[ii] - cdv[ii]);
        }
  #pragma unroll
        for (int db = 0; db < DB; ++db) {
          dva[kb][db] = mma16(adt[db], pg, dva[kb][db]);
          dka[kb][db] = mma16(aqt[db], dsv, dka[kb][db]);
        }
      }
    };
    for (int base = 0; base < nmine; base += kRound) {
      cnt = __builtin_amdgcn_readfirstlane(min(kRound, nmine - base));
      wave_sync();   // the previous round's row list and slots are no longer read
      for (int e = lane; e < cnt; e += 64) {
        const int item = wid + NWV * (base + e);
        rows[e] = (int)groups[s0 + item / qblocks] * g + 16 * (item % qblocks);
      }
      vm_drain();    // key/value fragments and row indices are in before the ring starts
      wave_sync();
      issue(0, ring0);
      issue(1, ring1);
      for (int i = 0; i < cnt; i += 3) {   // straight-line body
        step(i, ring0, ring2);
        step(i + 1, ring1, ring0);
        step(i + 2, ring2, ring1);
      }
      vm_drain();    // the repeats still in flight land before the slots are reused
    }
    // fixed-order sum of the waves' partials (NWV > 1): wave 0 accumulates waves 1, 2, ...,
    // one 16-key block at a time, through the (now idle) first two ring slots
    float* red0 = reinterpret_cast<float*>(ring0);
    float* red1 = reinterpret_cast<float*>(ring1);
    static_assert(NWV == 1 || 16 * HD * 4 <= NWV * SLOT * 2, "reduction buffer");
  #pragma unroll
    for (int kb = 0; kb < KBW; ++kb) {
      for (int w = 1; w < NWV; ++w) {
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
      const size_t off = ((size_t)bh * N + blk * ls + 16 * kb + r) * HD;
  #pragma unroll
      for (int db = 0; db < DB; ++db) {
        float* pk = dk + off + 16 * db + 4 * j;
        float* pv = dv + off + 16 * db + 4 * j;
        float4 ok4 = *reinterpret_cast<float4*>(pk), ov4 = *reinterpret_cast<float4*>(pv);
        f32x4 a = dka[kb][db] * scale, c = dva[kb][db];
        a[0] += ok4.x; a[1] += ok4.y; a[2] += ok4.z; a[3] += ok4.w;
        c[0] += ov4.x; c[1] += ov4.y; c[2] += ov4.z; c[3] += ov4.w;
        store4(pk, a, 1.0f);
        store4(pv, c, 1.0f);
      }
    }
  };
  if constexpr (NWV == 1) {
    block(xcd_grouped_block(N / ls).x);   // one head's blocks per XCD run
  } else {
    // persistent workgroups: each takes the blocks blockIdx.x + gridDim.x * t, reads their
    // item counts together, and walks the ones of this launch's size class in turn
    __shared__ int todo[64 * NWV];
    __shared__ int ntodo;
    const int qb = g >= 16 ? g / 16 : 1;
    for (long long base = blockIdx.x; base < nseg; base += (long long)gridDim.x * (64 * NWV)) {
      __syncthreads();   // the previous round's list is no longer read
      if (threadIdx.x == 0) ntodo = 0;
      __syncthreads();
      const long long sg = base + (long long)gridDim.x * threadIdx.x;
      if (sg < nseg) {
        const int nw = (seg_end[sg] - seg_start[sg]) * qb;
        // (the list's order varies from run to run; each block's result does not depend on it)
        if (nw >= min_items && nw <= max_items) todo[atomicAdd(&ntodo, 1)] = (int)(sg - base);
      }
      __syncthreads();
      const int cnt = ntodo;
      for (int e = 0; e < cnt; ++e) {
        block(base + (long long)todo[e]);
        __syncthreads();   // LDS slots and the reduction buffer are reused by the next block
      }
    }
  }
}

template <typename T, int HD, int KBW>
void launch_slc_kv(dim3 grid, hipStream_t st, const T* q, const T* k, const T* v, const T* dout,
                   const uint8_t* valid, const uint32_t* groups, const int* seg_start, const int* seg_end, QTerms qt,
                   int H, int N, int ls, int g, long long nseg, float sl2, float scale, float* dk, float* dv) {
  if constexpr (sizeof(T) == 2) {
    hipLaunchKernelGGL((slc_bwd_kv_dma_kernel<HD, KBW, 1>), grid, dim3(64), 0, st, q, k, v, dout, valid, groups,
                       seg_start, seg_end, qt, H, N, ls, g, nseg, sl2, scale, dk, dv, 1, kSlcLightItems);
    // persistent: one workgroup per CU; eight waves, or four where a wave holds four key
    // blocks (eight would not fit their registers)
    constexpr int NH = KBW >= 4 ? 4 : 8;
    const dim3 pgrid((unsigned)std::min<long long>(nseg, kSlcHeavyGroups));
    hipLaunchKernelGGL((slc_bwd_kv_dma_kernel<HD, KBW, NH>), pgrid, dim3(64 * NH), 0, st, q, k, v, dout, valid, groups,
                       seg_start, seg_end, qt, H, N, ls, g, nseg, sl2, scale, dk, dv, kSlcLightItems + 1,
                       std::numeric_limits<int>::max());
  } else {
    hipLaunchKernelGGL((slc_bwd_kv_kernel<T, HD, KBW>), grid, dim3(256), 0, st, q, k, v, dout, valid, groups,
                       seg_start, seg_end, qt, H, N, ls, g, nseg, sl2, scale, dk, dv);
  }
}

template <typename T, int HD>
hipError_t slc_kv_impl(const Dims& D, const BwdArgs& A, hipStream_t st) {
  const long long rows = D.rows();
  const float sl2 = D.scale * kLog2e;
  QTerms qslc{(const float4*)A.terms + 2 * rows};
  const long long nseg = (long long)D.B * D.H * (D.N / D.ls);
  const int kbw = D.ls / 16;
  const dim3 grid((unsigned)nseg);
  const T* q = (const T*)A.q;
  const T* k = (const T*)A.k;
  const T* v = (const T*)A.v;
  const T* dout = (const T*)A.dout;
  if (kbw == 1)
    launch_slc_kv<T, HD, 1>(grid, st, q, k, v, dout, A.valid, A.pair_groups, A.seg_start, A.seg_end, qslc, D.H, D.N,
                            D.ls, D.g, nseg, sl2, D.scale, A.dk, A.dv);
  else if (kbw == 2)
    launch_slc_kv<T, HD, 2>(grid, st, q, k, v, dout, A.valid, A.pair_groups, A.seg_start, A.seg_end, qslc, D.H, D.N,
                            D.ls, D.g, nseg, sl2, D.scale, A.dk, A.dv);
  else
    launch_slc_kv<T, HD, 4>(grid, st, q, k, v, dout, A.valid, A.pair_groups, A.seg_start, A.seg_end, qslc, D.H, D.N,
                            D.ls, D.g, nseg, sl2, D.scale, A.dk, A.dv);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bwd_stage(const Dims& D, const BwdArgs& A, BwdStage stage, hipStream_t st) {
  return BSA_DISPATCH(bwd_stage_impl, D, A, stage, st);
}

hipError_t launch_slc_csr(const Dims& D, const BwdArgs& A, hipStream_t st, const uint32_t** groups_out) {
  const long long total = (long long)D.B * D.H * (D.N / D.g) * D.k;
  const int nblk = D.N / D.ls;
  const long long nseg = (long long)D.B * D.H * nblk;
  const uint32_t sentinel = (uint32_t)nseg;
  int bits = 1;
  while ((1ll << bits) <= (long long)sentinel) ++bits;
  const int tid = timing_begin("bwd.slc_csr", st);
  hipLaunchKernelGGL(slc_pairs_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, A.sel, total, D.k,
                     D.N / D.g, nblk, sentinel, A.pair_keys, A.pair_vals);
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)((nseg + 255) / 256)), dim3(256), 0, st, A.seg_start, nseg, 0);
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)((nseg + 255) / 256)), dim3(256), 0, st, A.seg_end, nseg, 0);
  uint32_t* kout = nullptr;
  uint32_t* vout = nullptr;
  hipError_t e = launch_radix_sort_pairs(A.pair_keys, A.pair_vals, A.pair_keys_tmp, A.pair_vals_tmp, A.sort_hist,
                                         total, bits, &kout, &vout, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(seg_bounds_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, kout, total, sentinel,
                     A.seg_start, A.seg_end);
  timing_end(tid, st);
  *groups_out = vout;
  return hipGetLastError();
}

hipError_t launch_slc_kv(const Dims& D, const BwdArgs& A, const uint32_t* groups, hipStream_t st) {
  BwdArgs A2 = A;
  A2.pair_groups = groups;
  hipError_t r;
  BSA_PHASE("bwd.slc_kv", st, r = BSA_DISPATCH(slc_kv_impl, D, A2, st));
  return r;
}

}  // namespace bsa
