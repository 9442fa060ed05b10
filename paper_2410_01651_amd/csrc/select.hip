// Causal relevance scores and top-k without the score matrix (Eq. 1 of the
// method) for long sequences: the split select and its merge.
#include "gca_device.hpp"
#include "gca_launch.hpp"

#include <algorithm>
#include <type_traits>

namespace gca {
namespace {

// --------------------------------------- split causal select (no matrix) ----
//
// The work of a long causal selection is a triangle of (landmark row, key
// chunk) pairs.  It is cut into work items: a block of kSelRows rows against a
// part of the key tiles (kSelTile key chunks each) that the block reaches, the
// tiles of one item all of one class (tile index mod 8, one class per XCD, so
// that each XCD's L2 holds one eighth of the landmark keys).  Each item leaves
// the best k of its candidates for every one of its rows in the workspace, and
// a merge pass takes each row's best k over its lists: an exact top-k, since
// any member of a row's top k is among the best k of its own item.
//
// An item is one workgroup of 4 waves, two per CU; wave w owns 32 of the
// block's rows and keeps their landmark queries in registers as MFMA B operands
// (queries are the product's columns), so a lane holds, per 32-key tile, 16
// candidate scores of one row in registers and folds them into its own
// running best-k list; the two lanes of a row share their lists' thresholds
// once per tile, so that a candidate below the k-th best of either list is
// dropped with one compare.  Key tiles (32 keys x D columns) are staged in LDS
// by direct-to-LDS copies, two tiles deep.

template <typename T> struct SelMax;
template <> struct SelMax<__bf16> { static constexpr int kCh = 8; };  // D <= 512 in registers
template <> struct SelMax<float> { static constexpr int kCh = 4; };   // D <= 256
constexpr int kSelThreads = 256;
constexpr int kSelWaves = kSelThreads / 64;
static_assert(kSelWaves * 32 == kSelRows, "one 32-row column block per wave");

struct SelParams {
  uint32_t* gthr;  // per landmark row: the best published k-th score (order bits of a packed key), 0 = none
  int64_t nQ, nKV, tiles, blocks, items_per_class, parts_max, lists;
  int D, K, tpp, tpp_shift;  // tiles per part, a power of two (parts need no division)
  float scale;
  uint64_t seed;
};

// Key tiles row block r reaches (key chunks below its last row).
__device__ __forceinline__ int64_t sel_block_tiles(const SelParams& p, int64_t r) {
  const int64_t last = min((r + 1) * kSelRows - 1, p.nQ - 1);
  if (last < 1) return 0;
  return min((last - 1) / kSelTile + 1, p.tiles);
}
// Tiles of class x among the first nt; parts they form.
__device__ __forceinline__ int64_t sel_class_tiles(int64_t nt, int x) {
  return nt > x ? (nt - x + kSelClasses - 1) / kSelClasses : 0;
}

// NCH: 64-column chunks of the landmark width (D / 64), a compile-time count so
// that the chunks' fragment reads and products form one straight schedule.
template <typename T, int KM, bool GUMBEL, int NCH>
__global__ __launch_bounds__(kSelThreads, 2) void select_part_kernel(const T* __restrict__ lq,
                                                                     const T* __restrict__ lk,
                                                                     float* __restrict__ ls, int* __restrict__ lj,
                                                                     SelParams p) {
  constexpr int TILE = kSelTile * kD;  // one 64-column chunk of a key tile
  static_assert(NCH >= 1 && NCH <= SelMax<T>::kCh, "landmark width held in registers");
  __shared__ __attribute__((aligned(16))) T stage[2 * NCH * TILE];

  // block -> (retrieval slice, class, item); items of a class in order of
  // descending row block, so the longest items start first
  const int x = (int)(blockIdx.x % kSelClasses);
  const int64_t rest = blockIdx.x / kSelClasses;
  const int64_t bhr = rest / p.items_per_class;
  int64_t it = rest % p.items_per_class;
  int64_t r = p.blocks - 1, part = -1, ncls = 0;
  for (; r >= 0; --r) {
    ncls = sel_class_tiles(sel_block_tiles(p, r), x);
    const int64_t np = (ncls + p.tpp - 1) >> p.tpp_shift;
    if (it < np) {
      part = it;
      break;
    }
    it -= np;
  }
  if (part < 0) return;  // this class has fewer items
  const int nu = (int)min<int64_t>(p.tpp, ncls - part * p.tpp);  // tiles of this item
  auto tile_of = [&](int u) -> int64_t { return x + kSelClasses * (part * p.tpp + u); };

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hh = lane >> 5, l32 = lane & 31;
  const int64_t t0w = r * kSelRows + 32 * wave;  // this wave's first row
  const int64_t t = t0w + l32;                   // this lane's row
  const T* qrow = lq + (bhr * p.nQ + min(t, p.nQ - 1)) * p.D;
  Frag<T> qf[NCH][4];
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      qf[c][kb] = load_frag(qrow + c * kD + 16 * kb + 8 * hh);

  // copies: every wave copies its share of each 32 x 64 chunk of a tile; the
  // last key tile may hold fewer than 32 keys (rows past it repeat the last)
  const TileCopy<T, kSelWaves, kSelTile> cp_full(wave, lane, p.D, kSelTile);
  const int last_rows = (int)(p.nKV - (p.tiles - 1) * kSelTile);
  const TileCopy<T, kSelWaves, kSelTile> cp_last(wave, lane, p.D, last_rows);
  const T* kbase = lk + bhr * p.nKV * p.D;
  auto issue = [&](int u) __device__ {
    const int64_t j = tile_of(u);
    const T* src = kbase + j * kSelTile * p.D;
    T* dst = stage + (u & 1) * NCH * TILE;
    const bool last = j == p.tiles - 1;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      if (last) cp_last.issue(src + c * kD, dst + c * TILE);
      else cp_full.issue(src + c * kD, dst + c * TILE);
    }
  };

  TopKeys<KM> L;
  L.init();
  issue(0);
  for (int u = 0; u < nu; ++u) {
    wait_vmem<0>();
    block_barrier();  // tile u is in; every wave is done with the other slot
    if (u + 1 < nu) issue(u + 1);
    const int64_t j0 = tile_of(u) * kSelTile;  // first key chunk of the tile
    // wave-uniform: some (row, key) pair of this wave's block is a candidate
    if (j0 < t0w + 31 && t0w < p.nQ) {
      // the row's threshold: the better k-th best of its two lanes' lists and of
      // what the row's other items have published (each is the score of a
      // candidate beaten by k - 1 others, so a candidate below it cannot be in
      // the row's top k).  This lane pair publishes its own with an atomic
      // maximum, which returns the best published so far; a value read late is
      // only a weaker filter, never a wrong one.
      uint32_t pa, pb;
      pair32((uint32_t)(L.k[KM - 1] >> 32), pa, pb);
      const uint32_t own = pa > pb ? pa : pb;
      uint32_t pub = 0u;
      if (hh == 0 && t < p.nQ && own != 0u)
        pub = __hip_atomic_fetch_max(p.gthr + bhr * p.nQ + t, own, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const T* sK = stage + (u & 1) * NCH * TILE;
      // S^T of the tile's 32 keys against the wave's 32 rows
      auto half_scores = [&](int key0) __device__ {
        f32x16 a = zero16();
#pragma unroll
        for (int c = 0; c < NCH; ++c)
#pragma unroll
          for (int kb = 0; kb < 4; ++kb) mma32(a, lds_frag(sK + c * TILE, key0 + l32, 16 * kb + 8 * hh), qf[c][kb]);
        return a;
      };
      const f32x16 acc = half_scores(0);
      uint32_t qa, qb;
      pair32(pub, qa, qb);
      const uint32_t hi = max(own, max(qa, qb));   // the best threshold's score bits
      const float ts = hi == 0u ? -INFINITY : key_score((uint64_t)hi << 32);
      // full tile: every key below every row of the wave (and inside the keys)
      const bool full = j0 + kSelTile <= t0w && j0 + kSelTile <= p.nKV && t0w + 31 < p.nQ;
      // accumulator register i holds key 8 (i / 4) + 4 hh + i % 4 of its 32-key half
      // (four consecutive keys per group of four registers: one generator call
      // gives their Gumbel noise).  A half's 16 candidates are filtered against
      // the threshold into a bit mask; then every lane inserts its surviving
      // candidates one per round, so a round costs one insert for the wave
      // however many rows have a survivor, and the wave runs as many rounds as
      // its lane with the most survivors.
      auto fold_half = [&](f32x16 a, int half_key0) __device__ {
        uint32_t mask = 0u;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int64_t jg = j0 + half_key0 + 8 * g + 4 * hh;
          f32x4 nz = f32x4{0.f, 0.f, 0.f, 0.f};
          if constexpr (GUMBEL) nz = gumbel_noise4(p.seed, (uint32_t)bhr, (uint32_t)t, (uint32_t)(jg >> 2));
#pragma unroll
          for (int m = 0; m < 4; ++m) {
            a[4 * g + m] = a[4 * g + m] * p.scale + nz[m];
            mask |= (uint32_t)(a[4 * g + m] >= ts) << (4 * g + m);
          }
        }
        if (!full) {
          // keys at or past the row (and rows past the end) are not candidates
          const int64_t lim = t < p.nQ ? t - (j0 + half_key0 + 4 * hh) : 0;  // keys below the row, from this lane's first
          uint32_t okm = 0u;
#pragma unroll
          for (int i = 0; i < 16; ++i) okm |= (uint32_t)(8 * (i >> 2) + (i & 3) < lim) << i;
          mask &= okm;
        }
        while (__builtin_amdgcn_ballot_w64(mask != 0u)) {
          if (mask != 0u) {
            const int i = __builtin_ctz(mask);
            mask &= mask - 1u;
            // a[i] by a four-level select on the bits of i
            float v8[8], v4[4], v2[2];
#pragma unroll
            for (int e = 0; e < 8; ++e) v8[e] = (i & 1) ? a[2 * e + 1] : a[2 * e];
#pragma unroll
            for (int e = 0; e < 4; ++e) v4[e] = (i & 2) ? v8[2 * e + 1] : v8[2 * e];
#pragma unroll
            for (int e = 0; e < 2; ++e) v2[e] = (i & 4) ? v4[2 * e + 1] : v4[2 * e];
            const float v = (i & 8) ? v2[1] : v2[0];
            L.insert(pack_key(v, (int)(j0 + half_key0 + 8 * (i >> 2) + 4 * hh + (i & 3))));
          }
        }
      };
      fold_half(acc, 0);
    }
  }

  // the row's best k: the partner lane's list entries inserted into this lane's
  // (the two lanes hold disjoint keys, so the partner's entry is the one that
  // differs from this lane's; equal entries are both empty)
  uint64_t pk[KM];
#pragma unroll
  for (int e = 0; e < KM; ++e) {
    uint32_t la, lb, ha, hb;
    pair32((uint32_t)L.k[e], la, lb);
    pair32((uint32_t)(L.k[e] >> 32), ha, hb);
    const bool own_first = la == (uint32_t)L.k[e] && ha == (uint32_t)(L.k[e] >> 32);
    pk[e] = own_first ? ((uint64_t)hb << 32 | lb) : ((uint64_t)ha << 32 | la);
  }
#pragma unroll
  for (int e = 0; e < KM; ++e)
    if (pk[e] != 0) L.insert(pk[e]);
  if (hh == 0 && t < p.nQ) {
    const int64_t o = ((bhr * p.nQ + t) * p.lists + x * p.parts_max + part) * p.K;
#pragma unroll
    for (int e = 0; e < KM; ++e) {
      if (e < p.K) {
        const bool real = L.k[e] != 0;
        ls[o + e] = real ? key_score(L.k[e]) : -INFINITY;
        lj[o + e] = real ? key_chunk(L.k[e]) : -1;
      }
    }
  }
}

__global__ void sel_clear_kernel(uint32_t* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// One wave per landmark row: the best k over the row's lists, written in
// ascending chunk order (GUMBEL: the lists rank noisy scores; sel gets the
// chosen chunks' raw scores, recomputed from the landmark rows).
template <typename T, int KM, bool GUMBEL>
__global__ __launch_bounds__(256) void select_merge_kernel(const float* __restrict__ ls, const int* __restrict__ lj,
                                                           int32_t* __restrict__ idx, float* __restrict__ sel,
                                                           const T* __restrict__ lq, const T* __restrict__ lk,
                                                           int64_t rows, SelParams p) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int64_t t = row % p.nQ, bhr = row / p.nQ;
  const int64_t nt = sel_block_tiles(p, t / kSelRows);
  TopList<KM> L;
  L.init();
  const int64_t base = row * p.lists * p.K;
  // entry e of the row: class e / (parts_max K), part, rank
  const int64_t per_class = p.parts_max * p.K;
  for (int64_t e = lane; e < p.lists * p.K; e += 64) {
    const int x = (int)(e / per_class);
    const int64_t in_class = e % per_class;
    const int64_t parts = (sel_class_tiles(nt, x) + p.tpp - 1) >> p.tpp_shift;
    if (in_class / p.K < parts) {
      const int jj = lj[base + e];
      if (jj >= 0) L.insert(ls[base + e], jj);
    }
  }
  float ms;
  int mj, cnt;
  wave_merge(L, p.K, ms, mj, cnt);
  if constexpr (GUMBEL) {
    if (lane < cnt) ms = p.scale * dot_rows(lq + (bhr * p.nQ + t) * p.D, lk + (bhr * p.nKV + mj) * p.D, p.D);
  }
  const int rank = rank_by_chunk(mj, cnt);
  int32_t* io = idx + row * p.K;
  float* so = sel + row * p.K;
  if (lane < cnt) {
    io[rank] = mj;
    so[rank] = ms;
  } else if (lane < p.K) {
    io[lane] = -1;
    so[lane] = -INFINITY;
  }
}

template <typename T, int KM, bool GUMBEL, int NCH>
hipError_t launch_split_select_n(const Shape& s, const void* lq, const void* lk, int32_t* idx, float* sel, void* ws,
                               hipStream_t st) {
  const SelectPlan plan = select_plan(s);
  SelParams p;
  p.nQ = s.nQ;
  p.nKV = s.nKV;
  p.tiles = plan.tiles;
  p.blocks = plan.blocks;
  p.items_per_class = plan.items_per_class;
  p.parts_max = plan.parts_max;
  p.lists = plan.lists;
  p.D = s.D;
  p.K = s.topk;
  p.tpp = plan.tiles_per_part;
  p.tpp_shift = __builtin_ctz((unsigned)plan.tiles_per_part);
  p.scale = s.score_scale;
  p.seed = s.gumbel_seed;
  const int64_t BHr = (int64_t)s.B * s.Hr;
  const size_t n = (size_t)BHr * s.nQ * plan.lists * s.topk;
  float* ls = reinterpret_cast<float*>(ws);
  int* lj = reinterpret_cast<int*>(reinterpret_cast<char*>(ws) + align256(n * sizeof(float)));
  p.gthr = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(ws) + 2 * align256(n * sizeof(float)));
  const int64_t nrows = BHr * s.nQ;
  launch_kernel("sel_clear_kernel", sel_clear_kernel, dim3((unsigned)std::min<int64_t>((nrows + 255) / 256, 1024)),
                dim3(256), 0, st, p.gthr, nrows);
  const int64_t items = BHr * kSelClasses * plan.items_per_class;
  if (items > 0)
    launch_kernel("select_part_kernel", select_part_kernel<T, KM, GUMBEL, NCH>, dim3((unsigned)items),
                  dim3(kSelThreads), 0, st, (const T*)lq, (const T*)lk, ls, lj, p);
  const int64_t rows = BHr * s.nQ;
  launch_kernel("select_merge_kernel", select_merge_kernel<T, KM, GUMBEL>, dim3((unsigned)((rows + 3) / 4)),
                dim3(256), 0, st, ls, lj, idx, sel, (const T*)lq, (const T*)lk, rows, p);
  return take_launch_error();
}

template <typename T, int KM, bool GUMBEL>
hipError_t launch_split_select(const Shape& s, const void* lq, const void* lk, int32_t* idx, float* sel, void* ws,
                               hipStream_t st) {
  switch (s.D / kD) {
    case 1: return launch_split_select_n<T, KM, GUMBEL, 1>(s, lq, lk, idx, sel, ws, st);
    case 2: return launch_split_select_n<T, KM, GUMBEL, 2>(s, lq, lk, idx, sel, ws, st);
    case 3: return launch_split_select_n<T, KM, GUMBEL, 3>(s, lq, lk, idx, sel, ws, st);
    case 4: return launch_split_select_n<T, KM, GUMBEL, 4>(s, lq, lk, idx, sel, ws, st);
    default: break;
  }
  if constexpr (SelMax<T>::kCh > 4) {
    switch (s.D / kD) {
      case 5: return launch_split_select_n<T, KM, GUMBEL, 5>(s, lq, lk, idx, sel, ws, st);
      case 6: return launch_split_select_n<T, KM, GUMBEL, 6>(s, lq, lk, idx, sel, ws, st);
      case 7: return launch_split_select_n<T, KM, GUMBEL, 7>(s, lq, lk, idx, sel, ws, st);
      case 8: return launch_split_select_n<T, KM, GUMBEL, 8>(s, lq, lk, idx, sel, ws, st);
      default: break;
    }
  }
  return hipErrorInvalidValue;  // the plan keeps wider landmarks off this path
}

}  // namespace

hipError_t launch_fused_select(const Shape& s, const void* lmk_q, const void* lmk_k, int32_t* idx, float* sel,
                               void* ws, hipStream_t stream) {
  if (!select_plan(s).split) return launch_fused_rowblocks(s, lmk_q, lmk_k, idx, sel, stream);
  auto run = [&](auto tag, auto gumbel) {
    using T = decltype(tag);
    constexpr bool G = decltype(gumbel)::value;
    if (s.topk <= 8) return launch_split_select<T, 8, G>(s, lmk_q, lmk_k, idx, sel, ws, stream);
    return launch_split_select<T, 16, G>(s, lmk_q, lmk_k, idx, sel, ws, stream);
  };
  if (s.bf16) return s.gumbel ? run(__bf16{}, std::true_type{}) : run(__bf16{}, std::false_type{});
  return s.gumbel ? run(float{}, std::true_type{}) : run(float{}, std::false_type{});
}

}  // namespace gca
