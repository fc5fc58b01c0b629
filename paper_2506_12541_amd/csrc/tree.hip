// Ball-tree ordering of point clouds (the ordering Ball Tree Attention runs on,
// Section 2.1 and 2.2), and the row gather/scatter between point order and ball order.
//
// Construction: a node of capacity C holding the point set S splits on the axis of
// largest spread (float64 difference of float32 extremes, lowest axis on ties); its
// points ordered by (coordinate, index) are cut after ceil(|S|/2): left child in slots
// [0, C/2), right child in [C/2, C). The result depends only on node sets, so the GPU
// is free to use any partition that preserves them.
//
// GPU plan. The three per-axis orderings of every cloud are produced once by a stable
// LSD radix sort (8-bit digits). Each node then keeps, for every axis, its points
// sorted on that axis, stored at the node's own slot range. A split reads the extremes
// of each axis at the ends of the lists and the median at position ceil(n/2)-1 of the
// split axis; every list is then stably partitioned by "key <= median key", which keeps
// all three lists sorted in both children. Levels with nodes larger than 1024 slots run
// as three small kernels per level over all nodes; the last ten levels run inside one
// workgroup per 1024-slot node, entirely in LDS.
#include <map>
#include <mutex>

#include "common.hpp"
#include "kernels.hpp"

namespace bsa {
namespace {

constexpr int kSortThreads = 256;
constexpr int kSortItems = 8;
constexpr int kSortTile = kSortThreads * kSortItems;  // 2048 keys per workgroup
constexpr int kRadix = 256;                           // 8-bit digits (one per thread)
constexpr int kScanChunk = 8192;                      // counts scanned per workgroup
constexpr int kLocalScanTiles = 64;   // up to this many tiles, each scatter workgroup scans itself
constexpr int kPartTile = 2048;                       // slots per partition workgroup
constexpr int kBottom = 1024;                         // node size finished in LDS

__device__ __forceinline__ uint32_t ordered_key(float x) {
  x = x + 0.0f;  // -0.0 -> +0.0
  uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Real points in the node with index `node` among the nodes of capacity 2^log2c of one
// cloud: follow the root-to-node path, left children take the ceiling half.
__device__ __forceinline__ int node_count(int n_real, int log2_npad, int log2c, int node) {
  int cnt = n_real;
  for (int t = log2_npad - log2c - 1; t >= 0; --t)
    cnt = ((node >> t) & 1) ? (cnt >> 1) : ((cnt + 1) >> 1);
  return cnt;
}

__device__ __forceinline__ float coord(const float* pts, int dim, int g, int a) {
  return a < dim ? pts[(size_t)g * dim + a] : 0.0f;
}

// Block-wide exclusive scan of one value per thread (blockDim.x threads, <= 1024).
__device__ int block_exclusive_scan(int v, int* lds_tmp, int* total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = (blockDim.x + 63) >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) lds_tmp[wid] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < nw; ++w) { int t = lds_tmp[w]; lds_tmp[w] = run; run += t; }
    lds_tmp[nw] = run;
  }
  __syncthreads();
  int res = x - v + lds_tmp[wid];
  if (total) *total = lds_tmp[nw];
  __syncthreads();
  return res;
}

// ---- radix sort of (key, point) per axis; grid.y = axis ----
__global__ void __launch_bounds__(kSortThreads) sort_init_kernel(const float* pts, int dim, int m,
                                                                 uint32_t* keys, uint32_t* vals) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  int a = blockIdx.y;
  if (i >= m) return;
  keys[(size_t)a * m + i] = ordered_key(coord(pts, dim, i, a));
  vals[(size_t)a * m + i] = (uint32_t)i;
}

// 8-bit digits: passes 0-3 sort on the key, later passes on the cloud index (val / n_real).
__device__ __forceinline__ uint32_t sort_digit(uint32_t key, uint32_t val, int pass, int n_real) {
  return pass < 4 ? (key >> (8 * pass)) & 255u : ((val / (uint32_t)n_real) >> (8 * (pass - 4))) & 255u;
}

// Digit counts of one tile (kSortTile items, item i of the tile at it * 256 + thread),
// stored digit-major: hist[(a * 256 + d) * ntiles + tile].
__global__ void __launch_bounds__(kSortThreads) sort_hist_kernel(const uint32_t* keys, const uint32_t* vals,
                                                                 int m, int pass, int n_real, int ntiles,
                                                                 uint32_t* hist) {
  __shared__ uint32_t cnt[kRadix];
  const int a = blockIdx.y, tile = blockIdx.x;
  cnt[threadIdx.x] = 0;
  __syncthreads();
  const uint32_t* K = keys + (size_t)a * m;
  const uint32_t* V = vals + (size_t)a * m;
  // every item's loads first (one round trip), then the counts
  uint32_t kk[kSortItems], vv[kSortItems];
#pragma unroll
  for (int it = 0; it < kSortItems; ++it) {
    const int i = tile * kSortTile + it * kSortThreads + threadIdx.x;
    kk[it] = i < m ? K[i] : 0u;
    vv[it] = i < m && pass >= 4 ? V[i] : 0u;
  }
#pragma unroll
  for (int it = 0; it < kSortItems; ++it) {
    const int i = tile * kSortTile + it * kSortThreads + threadIdx.x;
    if (i < m) atomicAdd(&cnt[sort_digit(kk[it], vv[it], pass, n_real)], 1u);
  }
  __syncthreads();
  hist[((size_t)a * kRadix + threadIdx.x) * ntiles + tile] = cnt[threadIdx.x];
}

// Exclusive scan of the digit-major counts of each axis in chunks of kScanChunk entries:
// each workgroup scans one chunk in place and leaves the chunk total in sums.
__global__ void __launch_bounds__(1024) sort_scan_kernel(uint32_t* hist, int total, uint32_t* sums) {
  __shared__ int tmp[17];
  const int chunk = blockIdx.x, nchunks = gridDim.x;
  uint32_t* H = hist + (size_t)blockIdx.y * total + (size_t)chunk * kScanChunk;
  const int n = min(kScanChunk, total - chunk * kScanChunk);
  constexpr int per = kScanChunk / 1024;
  const int s = threadIdx.x * per;
  int sum = 0;
  for (int i = s; i < s + per && i < n; ++i) sum += (int)H[i];
  int all = 0;
  int run = block_exclusive_scan(sum, tmp, &all);
  for (int i = s; i < s + per && i < n; ++i) {
    int t = (int)H[i];
    H[i] = (uint32_t)run;
    run += t;
  }
  // a single chunk is already the whole scan: its offset is 0 (no chunk-total pass runs)
  if (threadIdx.x == 0) sums[(size_t)blockIdx.y * nchunks + chunk] = nchunks == 1 ? 0u : (uint32_t)all;
}

// Exclusive scan of the chunk totals of each axis (one workgroup per axis).
__global__ void __launch_bounds__(1024) sort_scan_sums_kernel(uint32_t* sums, int nchunks) {
  __shared__ int tmp[17];
  uint32_t* S = sums + (size_t)blockIdx.y * nchunks;
  const int per = (nchunks + 1023) / 1024;
  const int s = threadIdx.x * per;
  int sum = 0;
  for (int i = s; i < s + per && i < nchunks; ++i) sum += (int)S[i];
  int run = block_exclusive_scan(sum, tmp, nullptr);
  for (int i = s; i < s + per && i < nchunks; ++i) {
    int t = (int)S[i];
    S[i] = (uint32_t)run;
    run += t;
  }
}

// Stable scatter of one tile. Items are taken in index order, 256 per round: within a
// round, an item's rank among equal digits comes from eight ballots (lanes of its wave
// with the same digit and a lower lane id) plus the counts of the lower waves and of the
// earlier rounds, all kept per digit in LDS. sums == nullptr (few tiles): the tile's output
// starts come from the unscanned counts, each thread summing its digit's row of tiles and
// the workgroup scanning those totals over the digits (no scan launches).
__global__ void __launch_bounds__(kSortThreads) sort_scatter_kernel(const uint32_t* keys, const uint32_t* vals,
                                                                    uint32_t* keys_out, uint32_t* vals_out,
                                                                    int m, int pass, int n_real, int ntiles,
                                                                    const uint32_t* hist, const uint32_t* sums,
                                                                    int nchunks) {
  __shared__ uint32_t run[kRadix];            // items of each digit in earlier rounds
  __shared__ uint32_t base[kRadix];           // output start of each digit for this tile
  __shared__ uint32_t wc[kSortThreads / 64][kRadix];   // this round's count per wave and digit
  const int a = blockIdx.y, tile = blockIdx.x, t = threadIdx.x;
  const int lane = t & 63, wid = t >> 6;
  const uint32_t* K = keys + (size_t)a * m;
  const uint32_t* V = vals + (size_t)a * m;
  if (sums == nullptr) {
    __shared__ int tmp[kSortThreads / 64 + 1];
    const uint32_t* hd = hist + ((size_t)a * kRadix + t) * ntiles;   // digit t's counts over tiles
    uint32_t tot = 0, part = 0;
    for (int tl = 0; tl < ntiles; ++tl) {
      const uint32_t c = hd[tl];
      tot += c;
      part += tl < tile ? c : 0u;
    }
    base[t] = (uint32_t)block_exclusive_scan((int)tot, tmp, nullptr) + part;
    run[t] = 0;
  } else {
    const size_t e = (size_t)t * ntiles + tile;   // digit-major entry of (digit t, this tile)
    base[t] = hist[(size_t)a * kRadix * ntiles + e] + sums[(size_t)a * nchunks + e / kScanChunk];
    run[t] = 0;
  }
  const uint64_t below = (1ull << lane) - 1ull;
  uint32_t* KO = keys_out + (size_t)a * m;
  uint32_t* VO = vals_out + (size_t)a * m;
  // the tile's items are loaded before the rounds (one round trip instead of one per round)
  uint32_t kk[kSortItems], vv[kSortItems];
#pragma unroll
  for (int it = 0; it < kSortItems; ++it) {
    const int i = tile * kSortTile + it * kSortThreads + t;
    kk[it] = i < m ? K[i] : 0u;
    vv[it] = i < m ? V[i] : 0u;
  }
#pragma unroll
  for (int it = 0; it < kSortItems; ++it) {
    const int i = tile * kSortTile + it * kSortThreads + t;
    const bool ok = i < m;
    const uint32_t k = kk[it], v = vv[it];
    const uint32_t d = ok ? sort_digit(k, v, pass, n_real) : 0u;
#pragma unroll
    for (int w = 0; w < kSortThreads / 64; ++w) wc[w][t] = 0;
    uint64_t peers = __builtin_amdgcn_ballot_w64(ok);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const bool on = (d >> bit) & 1u;
      const uint64_t bb = __builtin_amdgcn_ballot_w64(on);
      peers &= on ? bb : ~bb;
    }
    const uint32_t rank = (uint32_t)__builtin_popcountll(peers & below);
    __syncthreads();   // wc cleared; run and base written
    if (ok && rank == 0) wc[wid][d] = (uint32_t)__builtin_popcountll(peers);
    __syncthreads();
    if (ok) {
      uint32_t off = base[d] + run[d] + rank;
      for (int w = 0; w < wid; ++w) off += wc[w][d];
      KO[off] = k;
      VO[off] = v;
    }
    __syncthreads();   // every item of the round has read run
    uint32_t add = 0;
#pragma unroll
    for (int w = 0; w < kSortThreads / 64; ++w) add += wc[w][t];
    run[t] += add;
  }
}

// Sorted position -> the axis list of its cloud, at slots [b*n_pad, b*n_pad + n_real).
__global__ void lists_init_kernel(const uint32_t* vals, int m, int n_real, int n_pad, int batch,
                                  int* lists) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int a = blockIdx.y;
  const size_t slots = (size_t)batch * n_pad;
  if (i >= slots) return;
  int b = (int)(i / n_pad), r = (int)(i % n_pad);
  lists[a * slots + i] = r < n_real ? (int)vals[(size_t)a * m + (size_t)b * n_real + r] : -1;
}

// ---- one top level: nodes of capacity 2^log2c (> kBottom) ----
struct NodeSplit {
  int axis;
  int med_idx;
  float med;
  int cnt;
};

// The split of node nd (of `slots` list slots in all): the axis of largest spread of its
// real points, and the median (the left child takes the ceiling half). Formed by the
// first nine threads of the workgroup together: each axis's two ends and its median
// candidate are loaded at once (two dependent round trips instead of eight), then thread
// 0 picks the axis. Every thread calls it; the split is returned to all of them.
__device__ NodeSplit node_split_block(const float* pts, int dim, int n_real, int n_pad, int log2_npad, int log2c,
                                     size_t slots, const int* lists, int nd) {
  __shared__ float ends[3][2];
  __shared__ int med_idx[3];
  __shared__ float med[3];
  __shared__ NodeSplit out;
  const int per_cloud = n_pad >> log2c;
  const int cnt = node_count(n_real, log2_npad, log2c, nd % per_cloud);
  const size_t start = (size_t)nd << log2c;
  const int t = threadIdx.x;
  if (cnt > 0 && t < 9) {
    if (t < 6) {   // axis t / 2: its lowest (t even) or highest (t odd) coordinate
      const int ax = t >> 1;
      ends[ax][t & 1] = coord(pts, dim, lists[ax * slots + start + ((t & 1) ? cnt - 1 : 0)], ax);
    } else {       // axis t - 6: its median
      const int ax = t - 6;
      const int g = lists[ax * slots + start + (cnt + 1) / 2 - 1];
      med_idx[ax] = g;
      med[ax] = coord(pts, dim, g, ax);
    }
  }
  __syncthreads();
  if (t == 0) {
    NodeSplit s{0, -1, 0.0f, cnt};
    if (cnt > 0) {
      double best = -1.0;
      for (int a = 0; a < 3; ++a) {
        const double sp = (double)ends[a][1] - (double)ends[a][0];
        if (sp > best) { best = sp; s.axis = a; }
      }
      s.med_idx = med_idx[s.axis];
      s.med = med[s.axis];
    }
    out = s;
  }
  __syncthreads();
  return out;
}

__device__ __forceinline__ bool goes_left(const float* pts, int dim, int g, const NodeSplit& s) {
  float c = coord(pts, dim, g, s.axis);
  return c < s.med || (c == s.med && g <= s.med_idx);
}

// Left-going points of one tile of one axis list. Each workgroup forms its node's split
// itself (a tile lies inside one node); the node's first tile of axis 0 stores it for the
// scatter.
__global__ void __launch_bounds__(256) part_count_kernel(const float* pts, int dim, int n_real, int n_pad,
                                                         int log2_npad, int log2c, const int* lists,
                                                         NodeSplit* splits, int tiles_per_list, int* tilecnt) {
  __shared__ int tmp[8];
  const int a = blockIdx.y, tile = blockIdx.x;
  const size_t slots = (size_t)tiles_per_list * kPartTile;
  const size_t s0 = (size_t)tile * kPartTile;
  const int nd = (int)(s0 >> log2c);
  const int off = (int)(s0 - ((size_t)nd << log2c));
  const NodeSplit sp = node_split_block(pts, dim, n_real, n_pad, log2_npad, log2c, slots, lists, nd);
  if (threadIdx.x == 0 && a == 0 && off == 0) splits[nd] = sp;
  // the tile's list entries first, then their coordinates (two round trips)
  int g[kPartTile / 256];
#pragma unroll
  for (int it = 0; it < kPartTile / 256; ++it) {
    const int i = threadIdx.x + 256 * it;
    g[it] = off + i < sp.cnt ? lists[a * slots + s0 + i] : -1;
  }
  int c = 0;
#pragma unroll
  for (int it = 0; it < kPartTile / 256; ++it) c += g[it] >= 0 && goes_left(pts, dim, g[it], sp);
  int total;
  block_exclusive_scan(c, tmp, &total);
  if (threadIdx.x == 0) tilecnt[a * tiles_per_list + tile] = total;
}

__global__ void __launch_bounds__(256) part_scatter_kernel(const float* pts, int dim, int log2c,
                                                           const int* lists, int* lists_out,
                                                           const NodeSplit* splits, int tiles_per_list,
                                                           const int* tilecnt) {
  __shared__ int tmp[8];
  const int a = blockIdx.y, tile = blockIdx.x;
  const size_t slots = (size_t)tiles_per_list * kPartTile;
  const size_t s0 = (size_t)tile * kPartTile;
  const int nd = (int)(s0 >> log2c);
  const NodeSplit sp = splits[nd];
  const size_t node_start = (size_t)nd << log2c;
  const int off = (int)(s0 - node_start);
  const int first_tile = (int)(node_start / kPartTile);
  // left-going elements in earlier tiles of this node
  int before = 0;
  for (int t = first_tile + (int)threadIdx.x; t < tile; t += 256) before += tilecnt[a * tiles_per_list + t];
  int left_before;
  block_exclusive_scan(before, tmp, &left_before);
  // each thread handles 8 consecutive slots
  constexpr int kItems = kPartTile / 256;
  int g[kItems];
  int f[kItems];
  int mine = 0;
#pragma unroll
  for (int it = 0; it < kItems; ++it) {
    int i = threadIdx.x * kItems + it;
    f[it] = -1;
    if (off + i < sp.cnt) {
      g[it] = lists[a * slots + s0 + i];
      f[it] = goes_left(pts, dim, g[it], sp) ? 1 : 0;
      mine += f[it];
    }
  }
  int lrank = block_exclusive_scan(mine, tmp, nullptr) + left_before;
  const int half = 1 << (log2c - 1);
#pragma unroll
  for (int it = 0; it < kItems; ++it) {
    if (f[it] < 0) continue;
    int pos_in_node = off + threadIdx.x * kItems + it;
    size_t dst;
    if (f[it]) {
      dst = node_start + lrank;
      ++lrank;
    } else {
      dst = node_start + half + (pos_in_node - lrank);
    }
    lists_out[a * slots + dst] = g[it];
  }
}

// ---- the last levels of one node of capacity T <= 1024, in LDS ----
// kBottomThreads threads per node, each owning a contiguous run of kBottomItems list slots
constexpr int kBottomThreads = 1024;
constexpr int kBottomItems = 3 * kBottom / kBottomThreads;
__global__ void __launch_bounds__(kBottomThreads) bottom_kernel(const float* pts, int dim, int n_real, int n_pad,
                                                     int log2_npad, int log2t, int nodes, const int* lists,
                                                     int* perm) {
  __shared__ float4 el[3 * kBottom];   // (x, y, z, point as int bits) per list slot
  __shared__ int sub_axis[kBottom / 2];
  __shared__ int sub_idx[kBottom / 2];
  __shared__ float sub_med[kBottom / 2];
  __shared__ int tmp[kBottomThreads / 64 + 1];
  const int T = 1 << log2t;
  const int nd = blockIdx.x;
  const size_t slots = (size_t)nodes << log2t;
  const size_t start = (size_t)nd << log2t;
  const int per_cloud = n_pad >> log2t;
  const int node_in_cloud = nd % per_cloud;
  const int cloud = nd / per_cloud;
  const int cnt0 = node_count(n_real, log2_npad, log2t, node_in_cloud);
  for (int i = threadIdx.x; i < 3 * T; i += kBottomThreads) {
    int a = i / T, r = i % T;
    float4 e = make_float4(0.f, 0.f, 0.f, __int_as_float(-1));
    if (r < cnt0) {
      int g = lists[a * slots + start + r];
      e = make_float4(coord(pts, dim, g, 0), coord(pts, dim, g, 1), coord(pts, dim, g, 2), __int_as_float(g));
    }
    el[i] = e;
  }
  __syncthreads();
  const int items = (3 * T + kBottomThreads - 1) / kBottomThreads;  // <= kBottomItems
  for (int log2c = log2t; log2c >= 1; --log2c) {
    const int C = 1 << log2c;
    const int nsub = T >> log2c;
    // split of every sub-node
    for (int s = threadIdx.x; s < nsub; s += kBottomThreads) {
      int cnt = node_count(n_real, log2_npad, log2c, node_in_cloud * nsub + s);
      int axis = 0, midx = -1;
      float med = 0.f;
      if (cnt > 0) {
        double best = -1.0;
        for (int a = 0; a < 3; ++a) {
          float4 lo = el[a * T + s * C], hi = el[a * T + s * C + cnt - 1];
          float l = a == 0 ? lo.x : (a == 1 ? lo.y : lo.z);
          float h = a == 0 ? hi.x : (a == 1 ? hi.y : hi.z);
          double sp = (double)h - (double)l;
          if (sp > best) { best = sp; axis = a; }
        }
        float4 me = el[axis * T + s * C + (cnt + 1) / 2 - 1];
        med = axis == 0 ? me.x : (axis == 1 ? me.y : me.z);
        midx = __float_as_int(me.w);
      }
      sub_axis[s] = axis;
      sub_idx[s] = midx;
      sub_med[s] = med;
    }
    __syncthreads();
    float4 e[kBottomItems];
    int f[kBottomItems];
    int mine = 0;
#pragma unroll
    for (int it = 0; it < kBottomItems; ++it) {
      f[it] = -1;
      int i = threadIdx.x * items + it;
      if (it < items && i < 3 * T) {
        e[it] = el[i];
        int g = __float_as_int(e[it].w);
        if (g >= 0) {
          int s = (i % T) >> log2c;
          int ax = sub_axis[s];
          float c = ax == 0 ? e[it].x : (ax == 1 ? e[it].y : e[it].z);
          f[it] = (c < sub_med[s] || (c == sub_med[s] && g <= sub_idx[s])) ? 1 : 0;
          mine += f[it];
        }
      }
    }
    // exclusive prefix of left flags over the concatenated lists; sub-node starts are
    // aligned to C, so the prefix at a sub-node start is subtracted below
    int pre = block_exclusive_scan(mine, tmp, nullptr);
    __shared__ int start_pref[3 * kBottom / 2];
    // record prefix at each sub-node start: the thread owning index (s*C) writes it
    {
      int run = pre;
#pragma unroll
      for (int it = 0; it < kBottomItems; ++it) {
        int i = threadIdx.x * items + it;
        if (it < items && i < 3 * T) {
          if ((i & (C - 1)) == 0) start_pref[i >> log2c] = run;
          run += f[it] > 0 ? 1 : 0;
        }
      }
    }
    __syncthreads();
    // all old values are in registers: rewrite the lists in place
    for (int i = threadIdx.x; i < 3 * T; i += kBottomThreads) el[i] = make_float4(0.f, 0.f, 0.f, __int_as_float(-1));
    __syncthreads();
    {
      int run = pre;
#pragma unroll
      for (int it = 0; it < kBottomItems; ++it) {
        int i = threadIdx.x * items + it;
        if (it < items && i < 3 * T && f[it] >= 0) {
          int sub_start = i & ~(C - 1);
          int lr = run - start_pref[i >> log2c];   // left flags before i in this sub-node
          int pos = i - sub_start;
          int dst = f[it] ? sub_start + lr : sub_start + C / 2 + (pos - lr);
          el[dst] = e[it];
        }
        if (it < items && i < 3 * T) run += f[it] > 0 ? 1 : 0;
      }
    }
    __syncthreads();
  }
  for (int r = threadIdx.x; r < T; r += kBottomThreads) {
    int g = __float_as_int(el[r].w);
    perm[start + r] = g >= 0 ? g - cloud * n_real : -1;
  }
}

// ---- row gather / scatter between point order and ball order ----
template <typename T>
__global__ void permute_kernel(const T* src, const int* perm, int n_real, int n_pad, int heads, int hd,
                               T* dst, uint8_t* valid, size_t total) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  // dst index [b, h, s, c]
  int c = (int)(i % hd);
  size_t r = i / hd;
  int s = (int)(r % n_pad);
  r /= n_pad;
  int h = (int)(r % heads);
  int b = (int)(r / heads);
  int p = perm[(size_t)b * n_pad + s];
  T val = T(0);
  if (p >= 0) val = src[((size_t)b * n_real + p) * heads * hd + (size_t)h * hd + c];
  dst[i] = val;
  if (valid && h == 0 && c == 0) valid[(size_t)b * n_pad + s] = p >= 0;
}

template <typename T>
__global__ void unpermute_kernel(const T* src, const int* perm, int n_real, int n_pad, int heads, int hd,
                                 T* dst, size_t total) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  int c = (int)(i % hd);
  size_t r = i / hd;
  int s = (int)(r % n_pad);
  r /= n_pad;
  int h = (int)(r % heads);
  int b = (int)(r / heads);
  int p = perm[(size_t)b * n_pad + s];
  if (p >= 0) dst[((size_t)b * n_real + p) * heads * hd + (size_t)h * hd + c] = src[i];
}

// 16-byte variant: one work item moves one 16-byte piece of a head row.
__global__ void permute16_kernel(const uint4* src, const int* perm, int n_real, int n_pad, int heads, int vpr,
                                 uint4* dst, uint8_t* valid, size_t total) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  int c = (int)(i % vpr);
  size_t r = i / vpr;
  int s = (int)(r % n_pad);
  r /= n_pad;
  int h = (int)(r % heads);
  int b = (int)(r / heads);
  int p = perm[(size_t)b * n_pad + s];
  uint4 val = make_uint4(0, 0, 0, 0);
  if (p >= 0) val = src[((size_t)b * n_real + p) * heads * vpr + (size_t)h * vpr + c];
  dst[i] = val;
  if (valid && h == 0 && c == 0) valid[(size_t)b * n_pad + s] = p >= 0;
}

__global__ void unpermute16_kernel(const uint4* src, const int* perm, int n_real, int n_pad, int heads, int vpr,
                                   uint4* dst, size_t total) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  int c = (int)(i % vpr);
  size_t r = i / vpr;
  int s = (int)(r % n_pad);
  r /= n_pad;
  int h = (int)(r % heads);
  int b = (int)(r / heads);
  int p = perm[(size_t)b * n_pad + s];
  if (p >= 0) dst[((size_t)b * n_real + p) * heads * vpr + (size_t)h * vpr + c] = src[i];
}

inline int ilog2(int64_t x) {
  int r = 0;
  while ((int64_t(1) << r) < x) ++r;
  return r;
}

}  // namespace

namespace {

constexpr size_t align256c(size_t x) { return (x + 255) & ~size_t(255); }

// Workspace bytes of the tree build over m real points in `slots` slots (all clouds); the
// carve-up in launch_build_tree follows the same order.
constexpr size_t tree_ws_bytes(size_t m, size_t slots) {
  const size_t ntiles = (m + kSortTile - 1) / kSortTile;
  return 4 * align256c(4 * 3 * m)                                            // keys and values, twice
         + align256c(4 * 3 * (size_t)kRadix * ntiles)                        // digit counts
         + align256c(4 * 3 * ((kRadix * ntiles + kScanChunk - 1) / kScanChunk))   // chunk totals
         + 2 * align256c(4 * 3 * slots)                                      // node lists, twice
         + align256c(sizeof(NodeSplit) * (slots / 2 + 1))
         + align256c(4 * 3 * (slots / kPartTile + 1));
}

// Scratch of the allocation-free tree build (bsa_build_ball_tree_noalloc): the workspace
// of up to kTreeScratchSlots slots, as one file-scope device array. Every term of
// tree_ws_bytes grows with m <= slots, so m = slots = the limit bounds every call. Each
// device holds its own copy; host code reaches it only through the address that
// hipGetSymbolAddress returns for the current device.
constexpr int64_t kTreeScratchSlots = int64_t(1) << 17;
constexpr size_t kTreeScratchBytes = tree_ws_bytes(kTreeScratchSlots, kTreeScratchSlots);
static __device__ __align__(256) unsigned char scratch[kTreeScratchBytes];

std::mutex g_scratch_mu;
std::map<int, void*> g_scratch_ptr;   // device -> address of its scratch array

}  // namespace

size_t tree_workspace_bytes(int64_t n_real, int64_t n_pad, int batch) {
  return tree_ws_bytes((size_t)batch * n_real, (size_t)batch * n_pad);
}

int64_t tree_scratch_slots() { return kTreeScratchSlots; }
size_t tree_scratch_bytes() { return kTreeScratchBytes; }

hipError_t tree_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  auto it = g_scratch_ptr.find(dev);
  if (it == g_scratch_ptr.end()) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));   // the current device's copy
    if (e != hipSuccess) return e;
    it = g_scratch_ptr.emplace(dev, p).first;
  }
  *ptr = it->second;
  return hipSuccess;
}

hipError_t launch_build_tree(const float* pts, int64_t n_real, int dim, int64_t n_pad, int batch,
                             int* perm, void* ws, hipStream_t st) {
  const size_t m = (size_t)batch * n_real;
  const size_t slots = (size_t)batch * n_pad;
  const int ntiles = (int)((m + kSortTile - 1) / kSortTile);
  char* p = (char*)ws;
  auto take = [&](size_t x) { char* r = p; p += (x + 255) & ~size_t(255); return r; };
  uint32_t* ka = (uint32_t*)take(4 * 3 * m);
  uint32_t* kb = (uint32_t*)take(4 * 3 * m);
  uint32_t* va = (uint32_t*)take(4 * 3 * m);
  uint32_t* vb = (uint32_t*)take(4 * 3 * m);
  uint32_t* hist = (uint32_t*)take(4 * 3 * (size_t)kRadix * ntiles);
  const int nchunks = (kRadix * ntiles + kScanChunk - 1) / kScanChunk;
  uint32_t* sums = (uint32_t*)take(4 * 3 * (size_t)nchunks);
  int* la = (int*)take(4 * 3 * slots);
  int* lb = (int*)take(4 * 3 * slots);
  NodeSplit* splits = (NodeSplit*)take(sizeof(NodeSplit) * (slots / 2 + 1));
  int* tilecnt = (int*)take(4 * 3 * (slots / kPartTile + 1));

  hipLaunchKernelGGL(sort_init_kernel, dim3((unsigned)((m + 255) / 256), 3), dim3(256), 0, st, pts, dim,
                     (int)m, ka, va);
  int passes = 4;
  for (int bits = 0; (1 << bits) < batch; bits += 8) ++passes;
  const bool local_scan = ntiles <= kLocalScanTiles;
  for (int pass = 0; pass < passes; ++pass) {
    hipLaunchKernelGGL(sort_hist_kernel, dim3(ntiles, 3), dim3(kSortThreads), 0, st, ka, va, (int)m, pass,
                       (int)n_real, ntiles, hist);
    if (!local_scan) {
      hipLaunchKernelGGL(sort_scan_kernel, dim3(nchunks, 3), dim3(1024), 0, st, hist, kRadix * ntiles, sums);
      if (nchunks > 1) hipLaunchKernelGGL(sort_scan_sums_kernel, dim3(1, 3), dim3(1024), 0, st, sums, nchunks);
    }
    hipLaunchKernelGGL(sort_scatter_kernel, dim3(ntiles, 3), dim3(kSortThreads), 0, st, ka, va, kb, vb,
                       (int)m, pass, (int)n_real, ntiles, hist, local_scan ? nullptr : sums, nchunks);
    std::swap(ka, kb);
    std::swap(va, vb);
  }
  hipLaunchKernelGGL(lists_init_kernel, dim3((unsigned)((slots + 255) / 256), 3), dim3(256), 0, st, va,
                     (int)m, (int)n_real, (int)n_pad, batch, la);
  const int log2_npad = ilog2(n_pad);
  const int log2t = log2_npad < 10 ? log2_npad : 10;
  for (int log2c = log2_npad; log2c > log2t; --log2c) {
    const int tiles = (int)(slots / kPartTile);
    hipLaunchKernelGGL(part_count_kernel, dim3(tiles, 3), dim3(256), 0, st, pts, dim, (int)n_real, (int)n_pad,
                       log2_npad, log2c, la, splits, tiles, tilecnt);
    hipLaunchKernelGGL(part_scatter_kernel, dim3(tiles, 3), dim3(256), 0, st, pts, dim, log2c, la, lb,
                       splits, tiles, tilecnt);
    std::swap(la, lb);
  }
  const int nodes = (int)(slots >> log2t);
  hipLaunchKernelGGL(bottom_kernel, dim3(nodes), dim3(kBottomThreads), 0, st, pts, dim, (int)n_real, (int)n_pad,
                     log2_npad, log2t, nodes, la, perm);
  return hipGetLastError();
}

size_t radix_sort_hist_words(long long n) {
  const size_t ntiles = (size_t)((n + kSortTile - 1) / kSortTile);
  return (size_t)kRadix * ntiles + (kRadix * ntiles + kScanChunk - 1) / kScanChunk;   // counts + chunk totals
}

hipError_t launch_radix_sort_pairs(uint32_t* keys, uint32_t* vals, uint32_t* keys_tmp, uint32_t* vals_tmp,
                                   uint32_t* hist, long long n, int bits, uint32_t** keys_out, uint32_t** vals_out,
                                   hipStream_t st) {
  const int ntiles = (int)((n + kSortTile - 1) / kSortTile);
  const int nchunks = (kRadix * ntiles + kScanChunk - 1) / kScanChunk;
  uint32_t* sums = hist + (size_t)kRadix * ntiles;
  const int passes = (bits + 7) / 8;  // key digits only (pass < 4)
  uint32_t *ka = keys, *va = vals, *kb = keys_tmp, *vb = vals_tmp;
  const bool local_scan = ntiles <= kLocalScanTiles;
  for (int pass = 0; pass < passes; ++pass) {
    hipLaunchKernelGGL(sort_hist_kernel, dim3(ntiles, 1), dim3(kSortThreads), 0, st, ka, va, (int)n, pass, 1, ntiles,
                       hist);
    if (!local_scan) {
      hipLaunchKernelGGL(sort_scan_kernel, dim3(nchunks, 1), dim3(1024), 0, st, hist, kRadix * ntiles, sums);
      if (nchunks > 1) hipLaunchKernelGGL(sort_scan_sums_kernel, dim3(1, 1), dim3(1024), 0, st, sums, nchunks);
    }
    hipLaunchKernelGGL(sort_scatter_kernel, dim3(ntiles, 1), dim3(kSortThreads), 0, st, ka, va, kb, vb, (int)n, pass,
                       1, ntiles, hist, local_scan ? nullptr : sums, nchunks);
    std::swap(ka, kb);
    std::swap(va, vb);
  }
  *keys_out = ka;
  *vals_out = va;
  return hipGetLastError();
}

hipError_t launch_permute(const void* src, const int* perm, int64_t n_real, int64_t n_pad, int batch,
                          int heads, int hd, int dtype, void* dst, uint8_t* valid, bool inverse,
                          hipStream_t st) {
  const size_t esz = dtype == 0 ? 4 : 2;
  if ((hd * esz) % 16 == 0) {
    const int vpr = (int)(hd * esz / 16);
    const size_t total = (size_t)batch * heads * n_pad * vpr;
    const unsigned blocks = (unsigned)((total + 255) / 256);
    if (!inverse)
      hipLaunchKernelGGL(permute16_kernel, dim3(blocks), dim3(256), 0, st, (const uint4*)src, perm, (int)n_real,
                         (int)n_pad, heads, vpr, (uint4*)dst, valid, total);
    else
      hipLaunchKernelGGL(unpermute16_kernel, dim3(blocks), dim3(256), 0, st, (const uint4*)src, perm, (int)n_real,
                         (int)n_pad, heads, vpr, (uint4*)dst, total);
    return hipGetLastError();
  }
  const size_t total = (size_t)batch * heads * n_pad * hd;
  const unsigned blocks = (unsigned)((total + 255) / 256);
  if (!inverse) {
    if (dtype == 0)
      hipLaunchKernelGGL(permute_kernel<float>, dim3(blocks), dim3(256), 0, st, (const float*)src, perm,
                         (int)n_real, (int)n_pad, heads, hd, (float*)dst, valid, total);
    else
      hipLaunchKernelGGL(permute_kernel<uint16_t>, dim3(blocks), dim3(256), 0, st, (const uint16_t*)src, perm,
                         (int)n_real, (int)n_pad, heads, hd, (uint16_t*)dst, valid, total);
  } else {
    if (dtype == 0)
      hipLaunchKernelGGL(unpermute_kernel<float>, dim3(blocks), dim3(256), 0, st, (const float*)src, perm,
                         (int)n_real, (int)n_pad, heads, hd, (float*)dst, total);
    else
      hipLaunchKernelGGL(unpermute_kernel<uint16_t>, dim3(blocks), dim3(256), 0, st, (const uint16_t*)src,
                         perm, (int)n_real, (int)n_pad, heads, hd, (uint16_t*)dst, total);
  }
  return hipGetLastError();
}

}  // namespace bsa
