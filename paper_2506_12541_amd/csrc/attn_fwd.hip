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
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "attn_common.hpp"

namespace bsa {
namespace {

// ---- dense kernel: ball branch (keys = own ball) and compressed branch (all tokens) ----

// Keys are staged 128 at a time (one pair of barriers) and consumed as two 64-key
// halves; the next 128 keys are loaded into registers while the current ones are used.
template <typename T, int HD, int QB, bool BALL, typename OT = T, bool LO = false>
__global__ void __launch_bounds__(256) dense_fwd_kernel(const T* q, const T* k, const T* v, const uint8_t* qvalid_all,
                                                        const uint8_t* kvalid_all, int H, int N, int nkeys_total,
                                                        int m, float sl2, OT* out, float* lse) {
  constexpr int kFT = sizeof(T) == 2 ? 128 : 64;  // keys per staged tile (LDS stays < 64 KB)
  constexpr int KSTR = HD + 16 / (int)sizeof(T);  // LDS row stride of K (elements)
  constexpr int VSTR = kFT + 4;                   // LDS row stride of V^T
  __shared__ __attribute__((aligned(16))) T ks[kFT * KSTR];
  __shared__ __attribute__((aligned(16))) T vt[HD * VSTR];
  __shared__ uint8_t kok[kFT];
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

  WaveAttn<T, HD, QB, LO> w;
  w.init();
  const int wq0 = q0 + wid * 16 * QB;
  load_q(w, q + (bh * N + wq0) * HD, lane);

  typedef TileIO<T, HD, kFT> IO;
  uint4 kreg[IO::RV];
  typename IO::V4 vreg[IO::TV][4];
  IO::load_rows(kreg, kh, 0, nkeys);
  IO::load_tr(vreg, vh, 0, nkeys);
  vm_drain();
  for (int t0 = 0; t0 < nkeys; t0 += kFT) {
    __syncthreads();
    IO::store_rows(kreg, ks, KSTR);
    IO::store_tr(vreg, vt, VSTR);
    if (threadIdx.x < kFT) {
      const int key = t0 + threadIdx.x;
      kok[threadIdx.x] = key < nkeys && (kval == nullptr || kval[key]);
    }
    __syncthreads();
    if (t0 + kFT < nkeys) {   // next keys in flight while these are used
      IO::load_rows(kreg, kh, t0 + kFT, nkeys);
      IO::load_tr(vreg, vh, t0 + kFT, nkeys);
    }
#pragma unroll
    for (int half = 0; half < kFT / kKT; ++half) {
      const int h0 = half * kKT;
      if (t0 + h0 >= nkeys) break;
      auto kfrag = [&](int kb, int c) { return load_chunk(&ks[(h0 + kb * 16 + r) * KSTR + 32 * c + 8 * j]); };
      auto vfrag = [&](int db, int kp) { return load_4x2(&vt[(16 * db + r) * VSTR + h0 + 32 * kp + 4 * j]); };
      if (kval == nullptr && t0 + h0 + kKT <= nkeys) {
        w.template tile<kKT / 16>(sl2, kfrag, vfrag, [](int, int, int) { return true; });
      } else {
        auto keyok = [&](int kb, int i, int) { return kok[h0 + kb * 16 + 4 * j + i] != 0; };
        w.template tile<kKT / 16>(sl2, kfrag, vfrag, keyok);
      }
    }
  }
  w.finish(lane, bh * N + wq0, out, lse, qval, wq0);
}

// bf16 variant: 64-key tiles filled by direct global->LDS loads (no staging registers),
// V^T fragments from transpose reads of the row-major V tile. Each iteration takes one tile
// through its scores, row maxima, exponentials and P V product in turn while the next
// tile's K and V load into the other buffers; each buffer is its own LDS object and the
// loop is unrolled by two, so the compiler can tell that loads in flight into one buffer
// do not alias reads of another. A wave's MFMA and VALU phases alternate, and with up to
// four waves per SIMD (128 registers at d = 64, QB = 2) the MFMA bursts of the other waves
// fill each wave's exponentials. (A software-pipelined form that formed the scores of tile
// t + 1 beside the exponentials of tile t held two tiles of scores, took up to 208
// registers, ran at two waves per SIMD and was 8% slower.) MASK = false: every key of the
// launch is real and the key count a multiple of 64 (no per-key select).
// LO: log-sum-exp rows only (the V tiles are not loaded; no output rows).
// PS: the keys are stored multiplied by sl2 (scores come out in the exponent's units, see
// WaveAttn); sl2 is then not applied again.
// LDS of the forward: K and V tiles and key-validity bytes, double buffered (each buffer
// its own object)
struct FwdLds {
  bf16_t *ks0, *ks1, *vs0, *vs1;
  uint8_t *ok0, *ok1;
};
#define BSA_FWD_LDS(L)                                                                   \
  __shared__ __attribute__((aligned(16))) bf16_t L##_ks0[kKT * HD], L##_ks1[kKT * HD]; \
  __shared__ __attribute__((aligned(16))) bf16_t L##_vs0[kKT * HD], L##_vs1[kKT * HD]; \
  __shared__ uint8_t L##_ok0[kKT], L##_ok1[kKT];                                        \
  const FwdLds L{L##_ks0, L##_ks1, L##_vs0, L##_vs1, L##_ok0, L##_ok1}

template <typename OT>
struct FwdArgs {
  const bf16_t *q, *k, *v;
  const uint8_t *qvalid_all, *kvalid_all;
  int H, N, nkeys_total, m;
  float sl2;
  OT* out;
  float* lse;
};

// One workgroup: `lin` is its linear id in a grid of shape `grid`.
template <int HD, int QB, int NW, bool BALL, typename OT, bool LO, bool MASK, bool PS>
__device__ __forceinline__ void fwd_dma_body(const FwdLds& L, dim3 grid, unsigned lin, const FwdArgs<OT>& a) {
  constexpr int kFT = kKT;
  constexpr int KB = kFT / 16;
  typedef WaveAttn<bf16_t, HD, QB, LO, PS> WA;
  typedef typename WA::CT CT;
  bf16_t *const ks0 = L.ks0, *const ks1 = L.ks1, *const vs0 = L.vs0, *const vs1 = L.vs1;
  uint8_t *const ok0 = L.ok0, *const ok1 = L.ok1;
  const bf16_t *const q = a.q, *const k = a.k, *const v = a.v;
  const uint8_t *const qvalid_all = a.qvalid_all, *const kvalid_all = a.kvalid_all;
  const int H = a.H, N = a.N, nkeys_total = a.nkeys_total, m = a.m;
  const float sl2 = a.sl2;
  OT* const out = a.out;
  float* const lse = a.lse;
  const int lane = threadIdx.x & 63, wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 15, j = lane >> 4;
  const dim3 blk = xcd_grouped_block_at(lin, grid, BALL ? m / (16 * QB * NW) : (int)grid.x);
  const int b = blk.z, h = blk.y;
  const long long bh = (long long)b * H + h;
  const int q0 = blk.x * (16 * QB * NW);
  const int nkeys = BALL ? m : nkeys_total;
  const int key0 = BALL ? (q0 / m) * m : 0;
  const bf16_t* kh = k + (bh * nkeys_total + key0) * HD;
  const bf16_t* vh = v + (bh * nkeys_total + key0) * HD;
  const uint8_t* kval = kvalid_all ? kvalid_all + (size_t)b * nkeys_total + key0 : nullptr;
  const uint8_t* qval = qvalid_all ? qvalid_all + (size_t)b * N : nullptr;
  const int nt = (nkeys + kFT - 1) / kFT;   // key tiles

  // K tile (and its key-validity bytes, read before the tile loads so that waiting for them
  // does not wait for the tile) / V tile of tile t. The tile past the end is loaded too (its
  // rows clamp to the last key; the buffer is free and nothing reads it): with the issue
  // under a branch the loop took 15 more registers, a wave per SIMD fewer.
  auto issue_k = [&](int t, bf16_t* kd, uint8_t* okd) {
    if constexpr (MASK) {
      uint8_t okv = 0;
      if (threadIdx.x < kFT) {
        const int key = t * kFT + threadIdx.x;
        okv = key < nkeys && (kval == nullptr || kval[key]);
      }
      dma_tile<HD, kFT, NW>(kd, kh, t * kFT, nkeys, wid, lane);
      if (threadIdx.x < kFT) okd[threadIdx.x] = okv;
    } else {   // whole tiles; a tile past the end reloads the last one
      dma_tile_full<HD, kFT, NW>(kd, kh + (size_t)(t < nt ? t : nt - 1) * kFT * HD, wid, lane);
    }
  };
  auto issue_v = [&](int t, bf16_t* vd) {
    if constexpr (!LO) {
      if constexpr (MASK)
        dma_tile<HD, kFT, NW>(vd, vh, t * kFT, nkeys, wid, lane);
      else
        dma_tile_full<HD, kFT, NW>(vd, vh + (size_t)(t < nt ? t : nt - 1) * kFT * HD, wid, lane);
    }
  };
  WA w;
  w.init();
  const int wq0 = q0 + wid * 16 * QB;
  float alpha[QB], delta[QB];

  auto kfrag_of = [&](const bf16_t* kt) {
    return [=](int kb, int c) { return lds_row_chunk<HD>(kt, kb * 16 + r, 4 * c + j); };
  };
  auto keyok_of = [&](const uint8_t* ok) {
    return [=](int kb, int i) { return ok[kb * 16 + 4 * j + i] != 0; };
  };
  // iteration t: LDS holds K(t) and V(t); the other buffers are free once every wave has
  // passed the barrier and take tile t + 1 while this one is computed
  auto step = [&](int t, const bf16_t* kc, const uint8_t* okc, const bf16_t* vc, bf16_t* kn, uint8_t* okn,
                  bf16_t* vn) {
    vm_drain();
    __syncthreads();
    issue_k(t + 1, kn, okn);
    issue_v(t + 1, vn);
    f32x4 s[QB][KB];
    w.template scores<KB>(s, kfrag_of(kc));
    if (w.template tile_max<KB, MASK>(s, sl2, keyok_of(okc), alpha, delta)) {
      w.rescale(alpha);   // rare: a query's maximum rose (wave-uniform)
      if constexpr (PS) w.template shift<KB>(s, delta);
    }
    CT pf[QB][KB / 2];
    w.template probs<KB>(s, sl2, pf);
    w.template pv<KB>(pf, [&](int db, int kp) { return lds_tr_chunk<HD>(vc, 32 * kp, 16 * db, lane); });
  };
  issue_k(0, ks0, ok0);
  issue_v(0, vs0);
  load_q(w, q + (bh * N + wq0) * HD, lane);
  for (int t = 0; t < nt; t += 2) {
    step(t, ks0, ok0, vs0, ks1, ok1, vs1);
    if (t + 1 < nt) step(t + 1, ks1, ok1, vs1, ks0, ok0, vs0);
  }
  vm_drain();   // the last step's loads (a repeat of the last tile, never read)
  w.finish(lane, bh * N + wq0, out, lse, qval, wq0);
}

// Unmasked launches are held to 128 registers (four waves per SIMD; no spills at d = 64).
template <int HD, int QB, int NW, bool BALL, typename OT = bf16_t, bool LO = false, bool MASK = true, bool PS = false>
__global__ void __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(MASK ? 1 : 4)))
dense_fwd_dma_kernel(FwdArgs<OT> a) {
  BSA_FWD_LDS(L);
  fwd_dma_body<HD, QB, NW, BALL, OT, LO, MASK, PS>(L, gridDim,
                                                   blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z), a);
}

// The compressed attention (prescaled keys, float32 rows) and the ball attention (bf16
// rows) of unmasked bf16 layers in one launch: the compressed workgroups first, then the
// ball workgroups, which fill the CUs that the compressed launch's last round leaves idle
// and overlap their HBM traffic with its MFMA work. Four waves per SIMD, as above.
template <int HD>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4)))
dense_fwd_pair_kernel(FwdArgs<float> cmp, dim3 cgrid, FwdArgs<bf16_t> ball, dim3 bgrid) {
  BSA_FWD_LDS(L);
  const unsigned ncmp = cgrid.x * cgrid.y * cgrid.z;
  if (blockIdx.x < ncmp)
    fwd_dma_body<HD, 2, 4, false, float, false, false, true>(L, cgrid, blockIdx.x, cmp);
  else
    fwd_dma_body<HD, 2, 4, true, bf16_t, false, false, false>(L, bgrid, blockIdx.x - ncmp, ball);
}

// ---- selection kernel: one wave = 16 queries; keys = the selected blocks of its group(s) ----
// The wave's key sequence is the concatenation of the blocks selected for the groups its
// 16 queries belong to (one group when g >= 16); a lane only accepts keys of its own
// group's blocks. Keys are walked in tiles of 32 (two 16-key sub-blocks, each inside one
// selected block since l' is a multiple of 16).

template <typename T, int HD, bool LO = false>
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
  wave_sync();   // LDS regions are per wave

  WaveAttn<T, HD, 1, LO> w;
  w.init();
  load_q(w, q + (bh * N + wq0) * HD, lane);
  vm_drain();

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
    wave_sync();   // LDS regions are per wave
    for (int e = lane; e < 8 * (HD / 8); e += 64) {
      const int kq = e / (HD / 8), dc = (e % (HD / 8)) * 8;
      const int en = ent[kq >> 2];
      const T* rows[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) rows[u] = en >= 0 ? vh + (size_t)((en & 0xFFFFFF) + 4 * (kq & 3) + u) * HD : nullptr;
      stage_vt(rows, dc, vt, VSTR, 4 * kq);
    }
    wave_sync();   // LDS regions are per wave
    auto kfrag = [&](int kb, int c) { return kf[kb][c]; };
    auto vfrag = [&](int db, int kp) { return load_4x2(&vt[(16 * db + r) * VSTR + 32 * kp + 4 * j]); };
    auto keyok = [&](int kb, int i, int) { return ok[kb][i]; };
    w.template tile<2>(sl2, kfrag, vfrag, keyok);
  }
  w.finish(lane, bh * N + wq0, out, lse, val, wq0);
}

// bf16 variant of the selection kernel. Each wave double-buffers its key tiles (the 32 K
// rows and 32 V rows of two sub-blocks) in LDS, filled by direct global->LDS loads one tile
// ahead; the two buffers are distinct LDS objects and the tile loop is unrolled by two with
// a straight-line body (tiles past the end are loaded from row 0 and masked). Key validity
// is gathered into 16-bit masks while the sub-block list is built, so no load other than
// the tile loads runs in the loop.
// LO: log-sum-exp rows only (the V tiles are not loaded; no output rows).
template <int HD, int NW, bool LO = false>
__global__ void __launch_bounds__(NW * 64) slc_fwd_dma_kernel(const bf16_t* q, const bf16_t* k, const bf16_t* v,
                                                              const uint8_t* valid_all, const int* sel, int H, int N,
                                                              int ls, int kk, int g, float sl2, bf16_t* out,
                                                              float* lse) {
  constexpr int TILE = 32 * HD;    // one 32-key tile
  constexpr int SLOT = 2 * TILE;   // K tile, V tile
  __shared__ __attribute__((aligned(16))) bf16_t buf0[NW * SLOT], buf1[NW * SLOT];
  __shared__ int sub_all[NW][kMaxSub];          // first token of each 16-key sub-block (or -1), group in bits 24+
  __shared__ uint32_t okm_all[NW][kMaxSub];     // bit t: key t of the sub-block is a real token
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
  WaveAttn<bf16_t, HD, 1, LO> w;
  w.init();
  load_q(w, q + (bh * N + wq0) * HD, lane);
  vm_drain();
  wave_sync();   // LDS regions are per wave

  const int nt = __builtin_amdgcn_readfirstlane((nsub + 1) / 2);   // 32-key tiles
  auto issue = [&](int t, bf16_t* slot) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int e = 2 * t + kb < nsub ? sub[2 * t + kb] : -1;
      const int row = e >= 0 ? (e & 0xFFFFFF) : 0;
      bf16_t* base = slot + wid * SLOT + kb * 16 * HD;
      dma_tile_full<HD, 16, 1>(base, kh + (size_t)row * HD, 0, lane);
      if constexpr (!LO) dma_tile_full<HD, 16, 1>(base + TILE, vh + (size_t)row * HD, 0, lane);
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
    auto kfrag = [&](int kb, int c) { return lds_row_chunk<HD>(kt, 16 * kb + r, 4 * c + j); };
    auto vfrag = [&](int db, int kp) { return lds_tr_chunk_nowait<HD>(vt, 32 * kp, 16 * db, lane); };
    auto keyok = [&](int kb, int i, int) { return ((m[kb] >> (4 * j + i)) & 1u) != 0; };
    // every key of both sub-blocks real and of every lane's group: no per-key select
    if (__builtin_amdgcn_ballot_w64((m[0] & m[1]) != 0xFFFFu) == 0)
      w.template tile<2, decltype(kfrag), decltype(vfrag), decltype(keyok), false>(sl2, kfrag, vfrag, keyok);
    else
      w.template tile<2>(sl2, kfrag, vfrag, keyok);
  };
  issue(0, buf0);
  for (int t = 0; t < nt; t += 2) {   // straight-line body
    step(t, buf0, buf1);
    step(t + 1, buf1, buf0);
  }
  vm_drain();   // the loads past the end have landed
  w.finish(lane, bh * N + wq0, out, lse, val, wq0);
}

// 16 bytes per thread (8 bf16 or 4 f32 channels of one row): one sigmoid per branch and row
// chunk, vector loads and stores. ob holds the ball and selection rows (storage type), oc
// the compressed branch's (float32).
template <typename T>
__global__ void gate_fwd_vec_kernel(const T* ob, const float* oc, const float* gate, const uint8_t* valid, int H,
                                    int N, int hd, long long per_branch, T* out) {
  constexpr int EPV = 16 / (int)sizeof(T);
  const long long v = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long i = v * EPV;
  if (i >= per_branch) return;
  const long long row = i / hd;      // (b*H + h)*N + n
  const int n = (int)(row % N);
  const int b = (int)(row / ((long long)H * N));
  float acc[EPV];
#pragma unroll
  for (int e = 0; e < EPV; ++e) acc[e] = 0.f;
  if (valid == nullptr || valid[(size_t)b * N + n]) {
    const float* gm = gate + ((size_t)b * N + n) * 3;
#pragma unroll
    for (int br = 0; br < 3; ++br) {
      const float sg = 1.0f / (1.0f + __expf(-gm[br]));
      if (br == 1) {
#pragma unroll
        for (int e = 0; e < EPV; e += 4) {
          const float4 f = *reinterpret_cast<const float4*>(oc + i + e);
          acc[e] += sg * f.x;
          acc[e + 1] += sg * f.y;
          acc[e + 2] += sg * f.z;
          acc[e + 3] += sg * f.w;
        }
        continue;
      }
      const uint4 u = *reinterpret_cast<const uint4*>(ob + (br / 2) * per_branch + i);
      const T* x = reinterpret_cast<const T*>(&u);
#pragma unroll
      for (int e = 0; e < EPV; ++e) acc[e] += sg * to_f32<T>(x[e]);
    }
  }
  uint4 o;
  T* y = reinterpret_cast<T*>(&o);
#pragma unroll
  for (int e = 0; e < EPV; ++e) y[e] = from_f32<T>(acc[e]);
  *reinterpret_cast<uint4*>(out + i) = o;
}

// bf16 layers take the direct-load kernel (NW waves of QB 16-query blocks per workgroup);
// f32 layers the register-staged one (4 waves).
// OT: type of the output rows (the storage type, or float32 for unrounded outputs).
// o == nullptr: log-sum-exp rows only (the same kernel without the value products, so the
// statistics equal those of the full launch bit for bit).
// PS: bf16 keys stored multiplied by sl2 (the compressed tokens; f32 layers keep them plain).
template <typename T, int HD, int QB, bool BALL, int NW = 4, typename OT = T, bool PS = false>
void launch_dense_fwd(dim3 grid, hipStream_t st, const void* q, const void* k, const void* v, const uint8_t* qvalid,
                      const uint8_t* kvalid, int H, int N, int nkeys_total, int m, float sl2, void* o, float* lse) {
  if constexpr (sizeof(T) == 2) {
    // every key real and whole 64-key tiles: no per-key select
    const bool mask = kvalid != nullptr || (BALL ? m : nkeys_total) % kKT != 0;
    const FwdArgs<OT> a{(const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v, qvalid, kvalid, H, N, nkeys_total, m,
                        sl2, (OT*)o, lse};
    const dim3 blk(64 * NW);
    if (o && mask)
      hipLaunchKernelGGL((dense_fwd_dma_kernel<HD, QB, NW, BALL, OT, false, true, PS>), grid, blk, 0, st, a);
    else if (o)
      hipLaunchKernelGGL((dense_fwd_dma_kernel<HD, QB, NW, BALL, OT, false, false, PS>), grid, blk, 0, st, a);
    else if (mask)
      hipLaunchKernelGGL((dense_fwd_dma_kernel<HD, QB, NW, BALL, OT, true, true, PS>), grid, blk, 0, st, a);
    else
      hipLaunchKernelGGL((dense_fwd_dma_kernel<HD, QB, NW, BALL, OT, true, false, PS>), grid, blk, 0, st, a);
  } else {
    if (o)
      hipLaunchKernelGGL((dense_fwd_kernel<T, HD, QB, BALL, OT>), grid, dim3(256), 0, st, (const T*)q, (const T*)k,
                         (const T*)v, qvalid, kvalid, H, N, nkeys_total, m, sl2, (OT*)o, lse);
    else
      hipLaunchKernelGGL((dense_fwd_kernel<T, HD, QB, BALL, OT, true>), grid, dim3(256), 0, st, (const T*)q,
                         (const T*)k, (const T*)v, qvalid, kvalid, H, N, nkeys_total, m, sl2, (OT*)o, lse);
  }
}

template <typename T, int HD>
hipError_t ball_impl(const Dims& D, const void* q, const void* k, const void* v, const uint8_t* valid, void* o,
                     float* lse, hipStream_t st) {
  const float sl2 = D.scale * kLog2e;
  if (D.m >= 128)
    launch_dense_fwd<T, HD, 2, true>(dim3(D.N / 128, D.H, D.B), st, q, k, v, valid, valid, D.H, D.N, D.N, D.m, sl2,
                                     o, lse);
  else
    launch_dense_fwd<T, HD, 1, true>(dim3(D.N / 64, D.H, D.B), st, q, k, v, valid, valid, D.H, D.N, D.N, D.m, sl2,
                                     o, lse);
  return hipGetLastError();
}

// The compressed branch keeps float32 output rows: the backward's softmax delta
// rowsum(dO o) is formed from them, and a delta error is shared by every compressed key of
// the query, so it would add up over the blocks in the MLP weight gradients.
template <typename T, int HD>
hipError_t cmp_impl(const Dims& D, const void* q, const void* kc, const void* vc, const uint8_t* valid,
                    const uint8_t* cvalid, float* o, float* lse, hipStream_t st) {
  const float sl2 = D.scale * kLog2e;
  if (D.N % 128 == 0)
    launch_dense_fwd<T, HD, 2, false, 4, float, true>(dim3(D.N / 128, D.H, D.B), st, q, kc, vc, valid, cvalid,
                                                      D.H, D.N, D.N / D.l, D.m, sl2, o, lse);
  else   // 64 token slots: one 64-query workgroup per head
    launch_dense_fwd<T, HD, 1, false, 4, float, true>(dim3(D.N / 64, D.H, D.B), st, q, kc, vc, valid, cvalid,
                                                      D.H, D.N, D.N / D.l, D.m, sl2, o, lse);
  return hipGetLastError();
}

// Ball and compressed attention of an unmasked bf16 layer in one launch (dense_fwd_pair_kernel).
template <typename T, int HD>
hipError_t ball_cmp_impl(const Dims& D, const void* q, const void* k, const void* v, const void* kc, const void* vc,
                         void* ob, float* lse_ball, float* ocmp, float* lse_cmp, hipStream_t st) {
  if constexpr (sizeof(T) == 2) {
    const float sl2 = D.scale * kLog2e;
    const FwdArgs<float> cmp{(const bf16_t*)q, (const bf16_t*)kc, (const bf16_t*)vc, nullptr, nullptr, D.H, D.N,
                             D.N / D.l, D.m, sl2, ocmp, lse_cmp};
    const FwdArgs<bf16_t> ball{(const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v, nullptr, nullptr, D.H, D.N, D.N,
                               D.m, sl2, (bf16_t*)ob, lse_ball};
    const dim3 g(D.N / 128, D.H, D.B);
    hipLaunchKernelGGL((dense_fwd_pair_kernel<HD>), dim3(2 * g.x * g.y * g.z), dim3(256), 0, st, cmp, g, ball, g);
    return hipGetLastError();
  }
  return hipErrorNotSupported;
}

// Group compression (Eq. 15): the coarse queries attend to the compressed tokens; rows are
// coarse queries [B, H, N/l, d], valid iff their block holds a real token. Outputs stay in
// float32: the backward forms its softmax delta from them.
template <typename T, int HD>
hipError_t cmp_coarse_impl(const Dims& D, const void* qc, const void* kc, const void* vc, const uint8_t* cvalid,
                           float* oc, float* lsec, hipStream_t st) {
  const float sl2 = D.scale * kLog2e;
  const int nct = D.N / D.l;
  if (nct % 128 == 0)
    launch_dense_fwd<T, HD, 2, false, 4, float, true>(dim3(nct / 128, D.H, D.B), st, qc, kc, vc, cvalid, cvalid,
                                                      D.H, nct, nct, D.m, sl2, oc, lsec);
  else
    launch_dense_fwd<T, HD, 1, false, 4, float, true>(dim3(nct / 64, D.H, D.B), st, qc, kc, vc, cvalid, cvalid,
                                                      D.H, nct, nct, D.m, sl2, oc, lsec);
  return hipGetLastError();
}

// The copy of Eq. 15: row n of the compression branch takes float32 coarse row n / l when
// slot n holds a real token; padding rows get zeros and LSE -inf. One thread per 16
// output bytes; ob == nullptr copies the log-sum-exp rows only.
__global__ void expand_coarse_kernel(const float* oc, const float* lsec, const uint8_t* valid, int H, int N, int l,
                                     int hd, long long rows, float* ob, float* lse) {
  constexpr int EPV = 4;
  const int per_row = hd / EPV;
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * per_row) return;
  const long long row = i / per_row;   // (b * H + h) * N + n
  const int c = (int)(i % per_row);
  const long long bh = row / N;
  const int n = (int)(row % N);
  const int b = (int)(bh / H);
  const bool ok = valid == nullptr || valid[(size_t)b * N + n] != 0;
  const long long crow = bh * (N / l) + n / l;
  if (ob == nullptr) {   // log-sum-exp rows only
    if (c == 0) lse[row] = ok ? lsec[crow] : kNegInf;
    return;
  }
  float4 f = make_float4(0.f, 0.f, 0.f, 0.f);
  if (ok) f = *reinterpret_cast<const float4*>(oc + crow * hd + c * EPV);
  *reinterpret_cast<float4*>(ob + row * hd + c * EPV) = f;
  if (c == 0) lse[row] = ok ? lsec[crow] : kNegInf;
}

template <typename T, int HD>
hipError_t slc_impl(const Dims& D, const void* q, const void* k, const void* v, const uint8_t* valid, const int* sel,
                    void* o, float* lse, hipStream_t st) {
  const float sl2 = D.scale * kLog2e;
  if constexpr (sizeof(T) == 2) {
    constexpr int NW = 2;
    if (o)
      hipLaunchKernelGGL((slc_fwd_dma_kernel<HD, NW>), dim3(D.N / (16 * NW), D.H, D.B), dim3(64 * NW), 0, st,
                         (const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v, valid, sel, D.H, D.N, D.ls, D.k, D.g,
                         sl2, (bf16_t*)o, lse);
    else
      hipLaunchKernelGGL((slc_fwd_dma_kernel<HD, NW, true>), dim3(D.N / (16 * NW), D.H, D.B), dim3(64 * NW), 0, st,
                         (const bf16_t*)q, (const bf16_t*)k, (const bf16_t*)v, valid, sel, D.H, D.N, D.ls, D.k, D.g,
                         sl2, (bf16_t*)o, lse);
  } else {
    if (o)
      hipLaunchKernelGGL((slc_fwd_kernel<T, HD>), dim3(D.N / 64, D.H, D.B), dim3(256), 0, st, (const T*)q,
                         (const T*)k, (const T*)v, valid, sel, D.H, D.N, D.ls, D.k, D.g, sl2, (T*)o, lse);
    else
      hipLaunchKernelGGL((slc_fwd_kernel<T, HD, true>), dim3(D.N / 64, D.H, D.B), dim3(256), 0, st, (const T*)q,
                         (const T*)k, (const T*)v, valid, sel, D.H, D.N, D.ls, D.k, D.g, sl2, (T*)o, lse);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_ball_fwd(const Dims& D, const void* q, const void* k, const void* v, const uint8_t* valid, void* o,
                           float* lse, hipStream_t st) {
  return BSA_DISPATCH(ball_impl, D, q, k, v, valid, o, lse, st);
}

hipError_t launch_cmp_fwd(const Dims& D, const void* q, const void* kc, const void* vc, const uint8_t* valid,
                          const uint8_t* cvalid, float* o, float* lse, hipStream_t st) {
  return BSA_DISPATCH(cmp_impl, D, q, kc, vc, valid, cvalid, o, lse, st);
}

bool ball_cmp_fwd_fits(const Dims& D) {
  const int nct = D.N / D.l;
  return D.bf16 && !D.gcmp && D.m >= 128 && D.m % kKT == 0 && D.N % 128 == 0 && nct % kKT == 0 &&
         (D.N / 128) * D.H * D.B % 8 == 0;
}

hipError_t launch_ball_cmp_fwd(const Dims& D, const void* q, const void* k, const void* v, const void* kc, const void* vc,
                               void* ob, float* lse_ball, float* ocmp, float* lse_cmp, hipStream_t st) {
  if (!ball_cmp_fwd_fits(D)) return hipErrorNotSupported;
  return BSA_DISPATCH(ball_cmp_impl, D, q, k, v, kc, vc, ob, lse_ball, ocmp, lse_cmp, st);
}

hipError_t launch_cmp_coarse_fwd(const Dims& D, const void* qc, const void* kc, const void* vc, const uint8_t* cvalid,
                                 float* oc, float* lsec, hipStream_t st) {
  return BSA_DISPATCH(cmp_coarse_impl, D, qc, kc, vc, cvalid, oc, lsec, st);
}

hipError_t launch_expand_coarse(const Dims& D, const float* oc, const float* lsec, const uint8_t* valid, float* ob,
                                float* lse, hipStream_t st) {
  const long long rows = D.rows();
  const long long per = rows * (D.d / 4);
  const unsigned grid = (unsigned)((per + 255) / 256);
  hipLaunchKernelGGL(expand_coarse_kernel, dim3(grid), dim3(256), 0, st, oc, lsec, valid, D.H, D.N, D.l, D.d, rows, ob,
                     lse);
  return hipGetLastError();
}

hipError_t launch_slc_fwd(const Dims& D, const void* q, const void* k, const void* v, const uint8_t* valid,
                          const int* sel, void* o, float* lse, hipStream_t st) {
  return BSA_DISPATCH(slc_impl, D, q, k, v, valid, sel, o, lse, st);
}

hipError_t launch_gate_fwd(const Dims& D, const void* ob, const float* ocmp, const float* gate, const uint8_t* valid,
                           void* o, hipStream_t st) {
  const long long per = D.rows() * D.d;
  if (D.bf16)
    hipLaunchKernelGGL(gate_fwd_vec_kernel<bf16_t>, dim3((unsigned)((per / 8 + 255) / 256)), dim3(256), 0, st,
                       (const bf16_t*)ob, ocmp, gate, valid, D.H, D.N, D.d, per, (bf16_t*)o);
  else
    hipLaunchKernelGGL(gate_fwd_vec_kernel<float>, dim3((unsigned)((per / 4 + 255) / 256)), dim3(256), 0, st,
                       (const float*)ob, ocmp, gate, valid, D.H, D.N, D.d, per, (float*)o);
  return hipGetLastError();
}

}  // namespace bsa
