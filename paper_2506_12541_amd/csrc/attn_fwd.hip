// Forward kernels of the three attention branches and the gate (Section 2.2):
//   ball attention        (Eq. 3)  each query attends to the real keys of its own ball;
//   compressed attention  (Eq. 5)  each query attends to every real compressed token;
//   selection attention   (Eq. 8)  each query attends to the tokens of the k* blocks
//                                  selected for its group (Eq. 10-12);
//   gate                  (Eq. 9)  o = sum_b sigmoid(gamma_b) * o_b, gamma per token.
// Scores use scale 1/sqrt(d) and no bias; a row without an eligible key outputs zeros
// and log-sum-exp -inf.
//
// All three branches share one wave-level flash-attention step (online softmax). It is
// written in the transposed form S^T = K Q^T, O^T = V^T P^T on 16x16 MFMA tiles: a
// lane owns one query column, so the probabilities produced by the first product are
// already laid out as the B operand of the second and never leave registers. V enters
// as V^T, which the kernels stage through LDS (transposing while storing).
#include "common.hpp"
#include "kernels.hpp"

namespace bsa {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();

// Two runs of 4 consecutive elements (at p and p + 16) as one 8-element chunk.
__device__ __forceinline__ bf16x8 load_4x2(const bf16_t* p) {
  uint2 a = *reinterpret_cast<const uint2*>(p);
  uint2 b = *reinterpret_cast<const uint2*>(p + 16);
  return __builtin_bit_cast(bf16x8, make_uint4(a.x, a.y, b.x, b.y));
}
__device__ __forceinline__ f32x8 load_4x2(const float* p) {
  float4 a = *reinterpret_cast<const float4*>(p);
  float4 b = *reinterpret_cast<const float4*>(p + 16);
  return f32x8{a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
}
__device__ __forceinline__ void store4(bf16_t* dst, f32x4 v, float sc) {
  uint32_t lo = (uint32_t)f2bf(v[0] * sc) | ((uint32_t)f2bf(v[1] * sc) << 16);
  uint32_t hi = (uint32_t)f2bf(v[2] * sc) | ((uint32_t)f2bf(v[3] * sc) << 16);
  *reinterpret_cast<uint2*>(dst) = make_uint2(lo, hi);
}
__device__ __forceinline__ void store4(float* dst, f32x4 v, float sc) {
  *reinterpret_cast<float4*>(dst) = make_float4(v[0] * sc, v[1] * sc, v[2] * sc, v[3] * sc);
}
// Write 4 consecutive keys of one dim of V^T (values of 4 rows, same column).
__device__ __forceinline__ void store_col4(bf16_t* dst, bf16_t a, bf16_t b, bf16_t c, bf16_t d) {
  *reinterpret_cast<uint2*>(dst) = make_uint2((uint32_t)a | ((uint32_t)b << 16), (uint32_t)c | ((uint32_t)d << 16));
}
__device__ __forceinline__ void store_col4(float* dst, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(dst) = make_float4(a, b, c, d);
}
// Stage 4 rows x 8 columns of V (row pointers may be null = zero rows) into V^T.
template <typename T>
__device__ __forceinline__ void stage_vt(const T* const (&rows)[4], int dc, T* vt, int vstr, int key_off) {
  T vals[4][8];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int x = 0; x < 8; ++x) vals[u][x] = rows[u] ? rows[u][dc + x] : T(0);
#pragma unroll
  for (int x = 0; x < 8; ++x)
    store_col4(vt + (dc + x) * vstr + key_off, vals[0][x], vals[1][x], vals[2][x], vals[3][x]);
}

// Online-softmax state of one wave over QB blocks of 16 queries.
template <typename T, int HD, int QB>
struct WaveAttn {
  static constexpr int NCH = HD / 32;  // chunks of the head dim
  static constexpr int DB = HD / 16;   // 16-wide dim blocks of O^T
  typedef typename Chunk<T>::type CT;
  CT qf[QB][NCH];
  float mx[QB];      // running max (log2 domain, scaled)
  float lsum[QB];    // this lane's partial row sum
  f32x4 o[QB][DB];

  __device__ void init() {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      mx[qb] = kNegInf;
      lsum[qb] = 0.f;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[qb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }

  // Process one tile of KB 16-key blocks (KB even). kfrag(kb, c) gives the A chunk of
  // key block kb, vfrag(db, kp) the A chunk of V^T for dim block db and key pair kp,
  // keyok(kb, i, qb) whether key 4j+i of block kb may be seen by this lane's query.
  template <int KB, typename KF, typename VF, typename OK>
  __device__ __forceinline__ void tile(float sl2, KF kfrag, VF vfrag, OK keyok) {
    f32x4 s[QB][KB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) s[qb][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        CT a = kfrag(kb, c);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) s[qb][kb] = mma(a, qf[qb][c], s[qb][kb]);
      }
    CT pf[QB][KB / 2];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float tmax = kNegInf;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float x = keyok(kb, i, qb) ? s[qb][kb][i] * sl2 : kNegInf;
          s[qb][kb][i] = x;
          tmax = fmaxf(tmax, x);
        }
      tmax = col_max(tmax);
      const float mnew = fmaxf(mx[qb], tmax);
      const float mref = mnew == kNegInf ? 0.f : mnew;
      const float alpha = fast_exp2(mx[qb] - mref);
      mx[qb] = mnew;
      float ps = 0.f;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float p = fast_exp2(s[qb][kb][i] - mref);
          s[qb][kb][i] = p;
          ps += p;
        }
      lsum[qb] = lsum[qb] * alpha + ps;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[qb][db] *= alpha;
#pragma unroll
      for (int kp = 0; kp < KB / 2; ++kp) {
        float v8[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          v8[i] = s[qb][2 * kp][i];
          v8[4 + i] = s[qb][2 * kp + 1][i];
        }
        pf[qb][kp] = make_chunk<T>(v8);
      }
    }
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int kp = 0; kp < KB / 2; ++kp) {
        CT a = vfrag(db, kp);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) o[qb][db] = mma(a, pf[qb][kp], o[qb][db]);
      }
  }

  // Normalise and store O rows (query q0 + 16 qb + r) and natural-log LSE.
  __device__ void finish(int lane, long long row0, T* out, float* lse, const uint8_t* qvalid, int qidx0) {
    const int r = lane & 15, j = lane >> 4;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float l = col_sum(lsum[qb]);
      const bool qok = qvalid == nullptr || qvalid[qidx0 + 16 * qb + r];
      const bool any = qok && l > 0.f;
      const float inv = any ? 1.0f / l : 0.f;
      const long long row = row0 + 16 * qb + r;
#pragma unroll
      for (int db = 0; db < DB; ++db) store4(out + row * HD + 16 * db + 4 * j, o[qb][db], inv);
      if (j == 0) lse[row] = any ? (mx[qb] + log2f(l)) * kLn2 : kNegInf;
    }
  }
};

template <typename T, int HD, int QB>
__device__ __forceinline__ void load_q(WaveAttn<T, HD, QB>& w, const T* qrow0, int lane) {
  const int r = lane & 15, j = lane >> 4;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int c = 0; c < WaveAttn<T, HD, QB>::NCH; ++c)
      w.qf[qb][c] = load_chunk(qrow0 + (size_t)(16 * qb + r) * HD + 32 * c + 8 * j);
}

// ---- dense kernel: ball branch (keys = own ball) and compressed branch (all tokens) ----
constexpr int kKT = 64;  // keys per LDS tile

template <typename T, int HD, int QB, bool BALL>
__global__ void __launch_bounds__(256) dense_fwd_kernel(const T* q, const T* k, const T* v, const uint8_t* qvalid_all,
                                                        const uint8_t* kvalid_all, int H, int N, int nkeys_total,
                                                        int m, float sl2, T* out, float* lse) {
  constexpr int KSTR = HD + 16 / (int)sizeof(T);  // LDS row stride of K (elements)
  constexpr int VSTR = kKT + 4;                   // LDS row stride of V^T
  constexpr int EPV = 16 / (int)sizeof(T);        // elements per 16-byte vector
  __shared__ __attribute__((aligned(16))) T ks[kKT * KSTR];
  __shared__ __attribute__((aligned(16))) T vt[HD * VSTR];
  __shared__ uint8_t kok[kKT];
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
  const uint8_t* qval = qvalid_all ? qvalid_all + (size_t)b * N : nullptr;

  WaveAttn<T, HD, QB> w;
  w.init();
  const int wq0 = q0 + wid * 16 * QB;
  load_q(w, q + (bh * N + wq0) * HD, lane);

  for (int t0 = 0; t0 < nkeys; t0 += kKT) {
    __syncthreads();
    for (int e = threadIdx.x; e < kKT * HD / EPV; e += 256) {
      const int row = e / (HD / EPV), col = (e % (HD / EPV)) * EPV;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (t0 + row < nkeys) val = *reinterpret_cast<const uint4*>(kh + (size_t)(t0 + row) * HD + col);
      *reinterpret_cast<uint4*>(&ks[row * KSTR + col]) = val;
    }
    for (int e = threadIdx.x; e < (kKT / 4) * (HD / 8); e += 256) {
      const int kq = e / (HD / 8), dc = (e % (HD / 8)) * 8;
      const T* rows[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int key = t0 + 4 * kq + u;
        rows[u] = key < nkeys ? vh + (size_t)key * HD : nullptr;
      }
      stage_vt<T>(rows, dc, vt, VSTR, 4 * kq);
    }
    if (threadIdx.x < kKT) {
      const int key = t0 + threadIdx.x;
      kok[threadIdx.x] = key < nkeys && (kval == nullptr || kval[key]);
    }
    __syncthreads();
    auto kfrag = [&](int kb, int c) { return load_chunk(&ks[(kb * 16 + r) * KSTR + 32 * c + 8 * j]); };
    auto vfrag = [&](int db, int kp) { return load_4x2(&vt[(16 * db + r) * VSTR + 32 * kp + 4 * j]); };
    auto keyok = [&](int kb, int i, int) { return kok[kb * 16 + 4 * j + i] != 0; };
    w.template tile<kKT / 16>(sl2, kfrag, vfrag, keyok);
  }
  w.finish(lane, bh * N + wq0, out, lse, qval, wq0);
}

// ---- selection kernel: one wave = 16 queries; keys = the selected blocks of its group(s) ----
// The wave's key sequence is the concatenation of the blocks selected for the groups its
// 16 queries belong to (one group when g >= 16); a lane only accepts keys of its own
// group's blocks. Keys are walked in tiles of 32 (two 16-key sub-blocks, each inside one
// selected block since l' is a multiple of 16).
constexpr int kMaxSub = 256;  // 16-key sub-blocks per wave (G * k* * l' / 16)

template <typename T, int HD>
__global__ void __launch_bounds__(256) slc_fwd_kernel(const T* q, const T* k, const T* v, const uint8_t* valid_all,
                                                      const int* sel, int H, int N, int ls, int kk, int g,
                                                      float sl2, T* out, float* lse) {
  constexpr int VSTR = 32 + 4;
  constexpr int NCH = HD / 32;
  __shared__ __attribute__((aligned(16))) T vt_all[4][HD * VSTR];
  __shared__ int sub_all[4][kMaxSub];   // first token of each 16-key sub-block (or -1), group in bits 24+
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
  T* vt = vt_all[wid];
  int* sub = sub_all[wid];

  const int nsub = G * kk * (ls / 16);
  for (int e = lane; e < nsub; e += 64) {
    const int slot = (e * 16) / ls;
    const int gi = slot / kk;
    const int id = selp[gi * kk + slot % kk];
    sub[e] = id < 0 ? -1 : ((gi << 24) | (id * ls + (e * 16) % ls));
  }
  __syncthreads();

  WaveAttn<T, HD, 1> w;
  w.init();
  load_q(w, q + (bh * N + wq0) * HD, lane);

  for (int sb0 = 0; sb0 < nsub; sb0 += 2) {
    const int e0 = sub[sb0];
    const int e1 = sb0 + 1 < nsub ? sub[sb0 + 1] : -1;
    const int ent[2] = {e0, e1};
    // this lane's A rows (key r of each sub-block) of K
    typename Chunk<T>::type kf[2][NCH];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        kf[kb][c] = zero_chunk(kf[kb][c]);
        if (ent[kb] >= 0) kf[kb][c] = load_chunk(kh + (size_t)((ent[kb] & 0xFFFFFF) + r) * HD + 32 * c + 8 * j);
      }
    // key validity of the score rows this lane holds: keys 4j+i of each sub-block
    bool ok[2][4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = ent[kb];
        const int tok = (e & 0xFFFFFF) + 4 * j + i;
        ok[kb][i] = e >= 0 && (e >> 24) == my_gi && (val == nullptr || val[tok]);
      }
    __syncthreads();
    for (int e = lane; e < 8 * (HD / 8); e += 64) {
      const int kq = e / (HD / 8), dc = (e % (HD / 8)) * 8;
      const int en = ent[kq >> 2];
      const T* rows[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) rows[u] = en >= 0 ? vh + (size_t)((en & 0xFFFFFF) + 4 * (kq & 3) + u) * HD : nullptr;
      stage_vt<T>(rows, dc, vt, VSTR, 4 * kq);
    }
    __syncthreads();
    auto kfrag = [&](int kb, int c) { return kf[kb][c]; };
    auto vfrag = [&](int db, int kp) { return load_4x2(&vt[(16 * db + r) * VSTR + 32 * kp + 4 * j]); };
    auto keyok = [&](int kb, int i, int) { return ok[kb][i]; };
    w.template tile<2>(sl2, kfrag, vfrag, keyok);
  }
  w.finish(lane, bh * N + wq0, out, lse, val, wq0);
}

template <typename T>
__global__ void gate_fwd_kernel(const T* ob, const float* gate, const uint8_t* valid, int H, int N, int hd,
                                long long per_branch, T* out) {
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= per_branch) return;
  long long row = i / hd;            // (b*H + h)*N + n
  int n = (int)(row % N);
  int b = (int)(row / ((long long)H * N));
  const float* gm = gate + ((size_t)b * N + n) * 3;
  float acc = 0.f;
  if (valid == nullptr || valid[(size_t)b * N + n]) {
#pragma unroll
    for (int br = 0; br < 3; ++br) {
      float s = 1.0f / (1.0f + __expf(-gm[br]));
      acc += s * to_f32<T>(ob[br * per_branch + i]);
    }
  }
  out[i] = from_f32<T>(acc);
}

template <typename T, int HD>
hipError_t ball_impl(const Dims& D, const void* q, const void* k, const void* v, const uint8_t* valid, void* o,
                     float* lse, hipStream_t st) {
  const float sl2 = D.scale * kLog2e;
  if (D.m >= 128) {
    dim3 grid(D.N / 128, D.H, D.B);
    hipLaunchKernelGGL((dense_fwd_kernel<T, HD, 2, true>), grid, dim3(256), 0, st, (const T*)q, (const T*)k,
                       (const T*)v, valid, valid, D.H, D.N, D.N, D.m, sl2, (T*)o, lse);
  } else {
    dim3 grid(D.N / 64, D.H, D.B);
    hipLaunchKernelGGL((dense_fwd_kernel<T, HD, 1, true>), grid, dim3(256), 0, st, (const T*)q, (const T*)k,
                       (const T*)v, valid, valid, D.H, D.N, D.N, D.m, sl2, (T*)o, lse);
  }
  return hipGetLastError();
}

template <typename T, int HD>
hipError_t cmp_impl(const Dims& D, const void* q, const void* kc, const void* vc, const uint8_t* valid,
                    const uint8_t* cvalid, void* o, float* lse, hipStream_t st) {
  const float sl2 = D.scale * kLog2e;
  dim3 grid(D.N / 128, D.H, D.B);
  hipLaunchKernelGGL((dense_fwd_kernel<T, HD, 2, false>), grid, dim3(256), 0, st, (const T*)q, (const T*)kc,
                     (const T*)vc, valid, cvalid, D.H, D.N, D.N / D.l, D.m, sl2, (T*)o, lse);
  return hipGetLastError();
}

template <typename T, int HD>
hipError_t slc_impl(const Dims& D, const void* q, const void* k, const void* v, const uint8_t* valid, const int* sel,
                    void* o, float* lse, hipStream_t st) {
  const float sl2 = D.scale * kLog2e;
  dim3 grid(D.N / 64, D.H, D.B);
  hipLaunchKernelGGL((slc_fwd_kernel<T, HD>), grid, dim3(256), 0, st, (const T*)q, (const T*)k, (const T*)v, valid,
                     sel, D.H, D.N, D.ls, D.k, D.g, sl2, (T*)o, lse);
  return hipGetLastError();
}

}  // namespace

#define BSA_DISPATCH(FN, ...)                                                              \
  (D.bf16 ? (D.d == 64 ? FN<bf16_t, 64>(__VA_ARGS__) : FN<bf16_t, 32>(__VA_ARGS__))       \
          : (D.d == 64 ? FN<float, 64>(__VA_ARGS__) : FN<float, 32>(__VA_ARGS__)))

hipError_t launch_ball_fwd(const Dims& D, const void* q, const void* k, const void* v, const uint8_t* valid, void* o,
                           float* lse, hipStream_t st) {
  return BSA_DISPATCH(ball_impl, D, q, k, v, valid, o, lse, st);
}

hipError_t launch_cmp_fwd(const Dims& D, const void* q, const void* kc, const void* vc, const uint8_t* valid,
                          const uint8_t* cvalid, void* o, float* lse, hipStream_t st) {
  return BSA_DISPATCH(cmp_impl, D, q, kc, vc, valid, cvalid, o, lse, st);
}

hipError_t launch_slc_fwd(const Dims& D, const void* q, const void* k, const void* v, const uint8_t* valid,
                          const int* sel, void* o, float* lse, hipStream_t st) {
  return BSA_DISPATCH(slc_impl, D, q, k, v, valid, sel, o, lse, st);
}

hipError_t launch_gate_fwd(const Dims& D, const void* ob, const float* gate, const uint8_t* valid, void* o,
                           hipStream_t st) {
  const long long per = D.rows() * D.d;
  const unsigned grid = (unsigned)((per + 255) / 256);
  if (D.bf16)
    hipLaunchKernelGGL(gate_fwd_kernel<bf16_t>, dim3(grid), dim3(256), 0, st, (const bf16_t*)ob, gate, valid, D.H, D.N,
                       D.d, per, (bf16_t*)o);
  else
    hipLaunchKernelGGL(gate_fwd_kernel<float>, dim3(grid), dim3(256), 0, st, (const float*)ob, gate, valid, D.H, D.N,
                       D.d, per, (float*)o);
  return hipGetLastError();
}

}  // namespace bsa
