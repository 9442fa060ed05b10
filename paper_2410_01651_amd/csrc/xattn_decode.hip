// Grouped cross attention for decode (Eq. 2-3 of the method for the one new
// query chunk of every (batch, head)), with the last step of its retrieval
// (Eq. 1 top-k) done in the same kernel.
//
// Decode has one work item per (batch, head), far too few to fill the chip, so
// the item is spread over its retrieved chunks instead of over query chunks:
// one workgroup per item, four pairs of waves, and the pairs take the item's
// valid slots side by side (two resident slots per pair for bf16, one for
// fp32; more than 8 or 4 slots take further rounds).  Within a pair each wave
// owns 32 of the chunk's 64 query tokens.  Because every retrieved chunk has
// its own softmax and the chunks are combined by the fusion weights, a slot's
// contribution w_s softmax(q K_s^T) V_s needs no information from the other
// slots: each wave accumulates its slots' weighted outputs in registers, and
// the four pairs' partial outputs are summed through LDS at the end.
//
// Selection: the scan leaves the best k of every wave range of the landmark
// keys; here each wave takes a share of those lists, keeps the lists headed by
// the k best maxima of its share and merges their entries, and wave 0 merges
// the waves' results into the row's top-k (merge_lists).  The slots are ordered
// by chunk index, as the selection step writes them.  For a caller that passes
// idx/sel, the same kernel reads them instead.
#include "gca_device.hpp"
#include "gca_launch.hpp"

#include <type_traits>

namespace gca {
namespace {

constexpr int kDecThreads = 512;
constexpr int kDecWaves = kDecThreads / 64;
constexpr int kDecPairs = kDecWaves / 2;

struct DecParams {
  const float* ls;  // scan lists (scores, chunks); null when idx/sel are inputs
  const int* lj;
  int64_t lists, pw;
  const void* q;
  const void* k;
  const void* v;
  int32_t* idx;
  float* sel;
  void* out;
  float* lse;
  float* w;
  int H, Hr, topk;
  int64_t nKV;
  float attn_scale;
  // Gumbel top-k: the lists rank noisy scores, so the chosen chunks' raw scores
  // are recomputed from the landmark rows
  int gumbel;
  const void* lmk_q;
  const void* lmk_k;
  int D;
  float score_scale;
};

template <typename T, bool OBO, bool MERGE, int KM>
__global__ __launch_bounds__(kDecThreads) void xattn_decode_kernel(DecParams p) {
  constexpr int TILE = kS * kD;
  constexpr bool kB16 = std::is_same<T, __bf16>::value;
  constexpr int SP = kB16 ? 2 : 1;  // resident slots per pair
  constexpr int kPerRound = kDecPairs * SP;
  constexpr uint32_t kTileB = TILE * sizeof(T), kRowB = kD * sizeof(T);
  // K and V tiles of every resident slot (128 KiB); reused for the partial outputs
  __shared__ __attribute__((aligned(16))) T ring[kDecPairs * SP * 2 * TILE];
  __shared__ float sMs[kDecWaves * 32];
  __shared__ int sMj[kDecWaves * 32];
  __shared__ int sCnt[kDecWaves];
  __shared__ int sSlot[32], sJc[32];  // the valid slots: slot, chunk, fusion weight
  __shared__ float sWc[32];
  __shared__ int sN;
  __shared__ uint32_t sValid;  // bit s: slot s is valid

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hh = lane >> 5;
  const int pair = wave >> 1, half = wave & 1;
  const int64_t wi = blockIdx.x;  // (batch, head)
  const int h = (int)(wi % p.H);
  const int64_t b = wi / p.H;
  const int64_t row = b * p.Hr + (p.Hr == 1 ? 0 : h);
  const int64_t row_off = row * p.topk;
  const bool owner = p.Hr != 1 || h == 0;  // writes the row's selection and weights
  const int K = p.topk;
  const int qi = 32 * half + (lane & 31);  // this lane's query token
  const int64_t tok0 = wi * kS;
  const float sc = p.attn_scale * kLog2e;
  const int cb = 16 * ((lane >> 4) & 1);

  // this wave's 32 queries: issued first, used after the selection
  Frag<T> qf[4];
  {
    const T* qr = reinterpret_cast<const T*>(p.q) + (tok0 + qi) * kD;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) qf[kb] = load_frag(qr + 16 * kb + 8 * hh);
  }

  // ---- selection: valid slots with their chunks and fusion weights (Eq. 2)
  if constexpr (MERGE) {
    float ms;
    int mj, cnt;
    merge_lists<KM, kDecWaves>(p.ls, p.lj, row, p.lists, p.pw, K, sMs, sMj, sCnt, ms, mj, cnt);
    if (wave == 0) {
      const bool valid = lane < cnt;
      const int rank = rank_by_chunk(mj, cnt);  // slots in ascending chunk order
      float mx;
      if (p.gumbel) {
        // raw scores of the chosen chunks: 8 lanes per chunk, each one eighth of
        // the D columns, summed over the 8 lanes
        const T* lq = reinterpret_cast<const T*>(p.lmk_q) + row * p.D;
        const int part = p.D / 8, sub = lane & 7;
        float raw = -INFINITY;
        for (int e0 = 0; e0 < cnt; e0 += 8) {
          const int e = e0 + (lane >> 3);
          const int je = __shfl(mj, e < cnt ? e : 0);
          const T* lk = reinterpret_cast<const T*>(p.lmk_k) + (row * p.nKV + (e < cnt ? je : 0)) * p.D;
          float acc = dot_rows(lq + sub * part, lk + sub * part, part);
          acc += dpp<kDppXor1>(acc);
          acc += dpp<kDppXor2>(acc);
          acc += dpp<kDppHalfMirror>(acc);
          const float mine = __shfl(acc, 8 * ((lane - e0) & 7));  // chunk `lane` of this group of 8
          if (lane >= e0 && lane < e0 + 8) raw = p.score_scale * mine;
        }
        ms = valid ? raw : -INFINITY;
        mx = max64(ms);
      } else {
        // the list is best first: lane 0 holds the maximum
        mx = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(ms)));
      }
      // the valid lanes (< cnt <= 32) all sit in the lower half
      const float e = valid ? expf(ms - mx) : 0.f;
      const float sum = sum32(e);
      const float wv = valid ? e / sum : 0.f;
      if (valid) {
        sSlot[rank] = rank;
        sJc[rank] = mj;
        sWc[rank] = wv;
      }
      if (lane == 0) {
        sN = cnt;
        sValid = cnt >= 32 ? 0xffffffffu : ((1u << cnt) - 1u);
      }
      if (owner && lane < K) {
        const int at = valid ? rank : lane;
        p.idx[row_off + at] = valid ? mj : -1;
        p.sel[row_off + at] = valid ? ms : -INFINITY;
        if (p.w) p.w[row_off + at] = wv;
      }
    }
  } else {
    if (wave == 0) {
      int j = -1;
      float sv = -INFINITY;
      if (lane < K) {
        j = p.idx[row_off + lane];
        sv = p.sel[row_off + lane];
      }
      const bool valid = lane < K && j >= 0 && j < p.nKV;
      const float mx = max64(valid ? sv : -INFINITY);
      const float e = valid ? expf(sv - mx) : 0.f;
      const float sum = sum64(e);
      const float wv = valid ? e / sum : 0.f;
      const uint64_t mask = __ballot(valid);
      if (valid) {
        const int rk = __popcll(mask & ((1ull << lane) - 1));
        sSlot[rk] = lane;
        sJc[rk] = j;
        sWc[rk] = wv;
      }
      if (lane == 0) {
        sN = __popcll(mask);
        sValid = (uint32_t)mask;
      }
      if (owner && p.w && lane < K) p.w[row_off + lane] = wv;
    }
  }
  __syncthreads();

  // ---- attention: the pairs take the valid slots kPerRound at a time
  const int n = sN;
  const TileCopy<T, 2> cp(half, lane);
  const T* const gk = reinterpret_cast<const T*>(p.k);
  const T* const gv = reinterpret_cast<const T*>(p.v);
  const int64_t kvb = wi * p.nKV * TILE;  // this (batch, head)'s key/value slice
  const lds_char* const lds0 = (const lds_char*)(ring);
  uint32_t kofs[4], vofs[2][2];
  {
    const uint32_t pb = (uint32_t)pair * SP * 2 * kTileB;
    const int s16 = lane & 15;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) kofs[kb] = pb + Swz<T>::off(lane & 31, 16 * kb + 8 * hh) * sizeof(T);
#pragma unroll
    for (int dh = 0; dh < 2; ++dh)
#pragma unroll
      for (int r8 = 0; r8 < 2; ++r8)
        vofs[dh][r8] =
            pb + kTileB + Swz<T>::off(8 * r8 + 4 * hh + (s16 >> 2), 32 * dh + cb + 4 * (s16 & 3)) * sizeof(T);
  }

  // slot s (chunk tiles in the pair's resident slot t) against this wave's queries
  auto compute = [&](int t, int s, float ws, f32x16& o0, f32x16& o1) __device__ {
    const uint32_t co = (uint32_t)t * 2 * kTileB;
    const T* sK = ring + (pair * SP + t) * (2 * TILE);
    const T* sV = sK + TILE;
    Frag<T> ka[8];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      if constexpr (kB16) {
        const lds_char* kp = lds0 + (kofs[kb] + co);
        ka[2 * kb] = lds_b128_at(kp);
        ka[2 * kb + 1] = lds_b128_at(kp + 32 * kRowB);
      } else {
        ka[2 * kb] = lds_frag(sK, lane & 31, 16 * kb + 8 * hh);
        ka[2 * kb + 1] = lds_frag(sK, 32 + (lane & 31), 16 * kb + 8 * hh);
      }
    }
    f32x16 st0 = zero16(), st1 = zero16();
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      mma32(st0, ka[2 * kb], qf[kb]);
      mma32(st1, ka[2 * kb + 1], qf[kb]);
    }
    Frag<T> va[8];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      if constexpr (kB16) {
        va[2 * kb] = lds_tr2(lds0 + (vofs[0][0] + co) + 16 * kb * kRowB, lds0 + (vofs[0][1] + co) + 16 * kb * kRowB);
        va[2 * kb + 1] =
            lds_tr2(lds0 + (vofs[1][0] + co) + 16 * kb * kRowB, lds0 + (vofs[1][1] + co) + 16 * kb * kRowB);
      } else {
        va[2 * kb] = lds_frag_t(sV, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, cb);
        va[2 * kb + 1] = lds_frag_t(sV, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, 32 + cb);
      }
    }
    // per-query softmax over the chunk's 64 keys (query = accumulator column)
    float mx = max_xor32(max_of(st0, st1)) * sc;
    if (OBO) mx = fmaxf(mx, 0.f);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      st0[i] = __builtin_amdgcn_exp2f(fmaf(st0[i], sc, -mx));
      st1[i] = __builtin_amdgcn_exp2f(fmaf(st1[i], sc, -mx));
    }
    float sum = st0[0] + st1[0];
#pragma unroll
    for (int i = 1; i < 16; ++i) sum += st0[i] + st1[i];
    sum = sum_xor32(sum);
    if (OBO) sum += __builtin_amdgcn_exp2f(-mx);
    if (p.lse && hh == 0) p.lse[(tok0 + qi) * K + s] = (mx + __builtin_amdgcn_logf(sum)) * kLn2;
    const float coef = ws * __builtin_amdgcn_rcpf(sum);
    Frag<T> pf[4];
    frag_from_acc(pf[0], st0, 0, coef);
    frag_from_acc(pf[1], st0, 1, coef);
    frag_from_acc(pf[2], st1, 0, coef);
    frag_from_acc(pf[3], st1, 1, coef);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      mma32(o0, va[2 * kb], pf[kb]);
      mma32(o1, va[2 * kb + 1], pf[kb]);
    }
  };

  // Each round: copy the pair's slots, then compute the first as soon as its
  // tiles are in (the second slot's copies still in flight).  Only the tile
  // copies are outstanding while they are waited for.
  constexpr int kSlotLoads = 2 * TileCopy<T, 2>::kN;  // one wave's copies for one slot
  f32x16 o0 = zero16(), o1 = zero16();
  for (int r0 = 0; r0 < n; r0 += kPerRound) {
    if (r0 > 0) block_barrier();  // the last round's tiles have been read
    wait_vmem<0>();
    const int i0 = r0 + pair * SP;
#pragma unroll
    for (int t = 0; t < SP; ++t) {
      if (i0 + t < n) {
        int j = sJc[i0 + t];
        j = min(max(j, 0), (int)p.nKV - 1);  // valid chunks only; never copy outside the slice
        T* dst = ring + (pair * SP + t) * (2 * TILE);
        cp.issue(gk + kvb + (int64_t)j * TILE, dst);
        cp.issue(gv + kvb + (int64_t)j * TILE, dst + TILE);
      }
    }
    if (SP == 2 && i0 + 1 < n)
      wait_vmem<kSlotLoads>();
    else
      wait_vmem<0>();
    block_barrier();
    if (i0 < n) compute(0, sSlot[i0], sWc[i0], o0, o1);
    if constexpr (SP == 2) {
      wait_vmem<0>();
      block_barrier();
      if (i0 + 1 < n) compute(1, sSlot[i0 + 1], sWc[i0 + 1], o0, o1);
    }
  }

  // slots with no chunk
  if (p.lse && n < K) {
    const uint32_t vm = sValid;
    for (int e = tid; e < kS * K; e += kDecThreads) {
      const int rr = e / K, s = e - rr * K;
      if (!((vm >> s) & 1u)) p.lse[(tok0 + rr) * K + s] = -INFINITY;
    }
  }

  // ---- sum the pairs' partial outputs through LDS: part[pair][row][16 float4
  // blocks], block c of row r stored at c ^ (r mod 16)
  block_barrier();
  float* part = reinterpret_cast<float*>(ring);
  {
    const int sw = qi & 15;
    float* pr = part + (pair * kS + qi) * kD;
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      *reinterpret_cast<f32x4*>(pr + 4 * ((2 * gq + hh) ^ sw)) =
          f32x4{o0[4 * gq], o0[4 * gq + 1], o0[4 * gq + 2], o0[4 * gq + 3]};
      *reinterpret_cast<f32x4*>(pr + 4 * ((8 + 2 * gq + hh) ^ sw)) =
          f32x4{o1[4 * gq], o1[4 * gq + 1], o1[4 * gq + 2], o1[4 * gq + 3]};
    }
  }
  __syncthreads();
  {
    const int rr = tid >> 3;  // output row; 8 threads per row, two 4-column blocks each
    T* orow = reinterpret_cast<T*>(p.out) + (tok0 + rr) * kD;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int c = 2 * (tid & 7) + e;
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int pp = 0; pp < kDecPairs; ++pp)
        acc += *reinterpret_cast<const f32x4*>(part + (pp * kS + rr) * kD + 4 * (c ^ (rr & 15)));
      store4(orow + 4 * c, acc[0], acc[1], acc[2], acc[3]);
    }
  }
}

template <typename T, bool OBO>
hipError_t launch_dec_t(const Shape& s, const DecParams& p, hipStream_t st) {
  const dim3 grid((unsigned)((int64_t)s.B * s.H)), block(kDecThreads);
  if (p.ls) {
    if (s.topk <= 8)
      launch_kernel("xattn_decode_kernel", xattn_decode_kernel<T, OBO, true, 8>, grid, block, 0, st, p);
    else if (s.topk <= 16)
      launch_kernel("xattn_decode_kernel", xattn_decode_kernel<T, OBO, true, 16>, grid, block, 0, st, p);
    else
      launch_kernel("xattn_decode_kernel", xattn_decode_kernel<T, OBO, true, 32>, grid, block, 0, st, p);
  } else {
    launch_kernel("xattn_decode_kernel", xattn_decode_kernel<T, OBO, false, 8>, grid, block, 0, st, p);
  }
  return take_launch_error();
}

}  // namespace

hipError_t launch_xattn_decode(const Shape& s, const float* list_s, const int* list_j, const void* q,
                               const void* k, const void* v, int32_t* idx, float* sel, void* out, float* lse,
                               float* w, const void* lmk_q, const void* lmk_k, hipStream_t stream) {
  DecParams p;
  p.ls = list_s;
  p.lj = list_j;
  const DecodePlan plan = decode_plan(s);
  p.lists = plan.lists;
  p.pw = plan.pw;
  p.q = q; p.k = k; p.v = v;
  p.idx = idx; p.sel = sel;
  p.out = out; p.lse = lse; p.w = w;
  p.H = s.H; p.Hr = s.Hr; p.topk = s.topk;
  p.nKV = s.nKV;
  p.attn_scale = s.attn_scale;
  p.gumbel = list_s != nullptr && s.gumbel;
  p.lmk_q = lmk_q;
  p.lmk_k = lmk_k;
  p.D = s.D;
  p.score_scale = s.score_scale;
  if (s.bf16)
    return s.off_by_one ? launch_dec_t<__bf16, true>(s, p, stream) : launch_dec_t<__bf16, false>(s, p, stream);
  return s.off_by_one ? launch_dec_t<float, true>(s, p, stream) : launch_dec_t<float, false>(s, p, stream);
}

}  // namespace gca
