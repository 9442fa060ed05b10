// Grouped cross attention forward (Eq. 2-3 of the method; Algorithm 1 in the
// appendix is its tiled form).
//
// Persistent workgroups of one wave pair, four per CU: each pair is a stream of
// (batch, head, query chunk) work items, and within a pair each wave owns 32 of
// the chunk's 64 query tokens and keeps their Q fragments in registers.  A pair
// takes its chunk's retrieved chunks one per round; their keys and values stream
// through the pair's two LDS ring slots, filled by asynchronous direct-to-LDS
// copies one round ahead of the compute (two waves per SIMD hide each other's
// MFMA, LDS and cross-lane latencies).  For every retrieved chunk (slot) a wave
// computes S^T = K Q^T on the matrix cores, takes each query's softmax over the
// 64 keys (one retrieved chunk is exactly one tile, so no running rescale is
// needed), folds the fusion weight w_s / l_s into P, and accumulates
// O^T += V^T (w_s P_s)^T in registers; at the end of the chunk each wave stores
// its rows.  The per-chunk outputs O'_s of Algorithm 1 are never written; the
// log-sum-exp of every (row, slot) is.
//
// Computing the transposed products keeps every query's statistics inside one
// lane (query = accumulator column): the softmax needs one cross-lane step, and
// the probability tile feeds the PV product straight from registers.  V^T
// fragments come from the row-major V tile through LDS transpose reads.
//
// With an LMK row per chunk (S + 1 query rows), the 65th row meets the same
// tiles: one wave per slot (the waves alternate) takes it as a vector against
// the K and V^T fragments it already holds, with one key per lane for the
// softmax, and the waves' partial outputs are added through LDS at the end of
// the chunk.
#include "gca_device.hpp"
#include "gca_launch.hpp"

#include <type_traits>

namespace gca {
namespace {

// wave pairs per workgroup: one, so that a round's barrier couples only the two
// waves that share a ring; four workgroups per CU
constexpr int kPairs = 1;
constexpr int kThreads = 128 * kPairs;
constexpr int kWgPerCu = 4 / kPairs;

struct FwdParams {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* idx;
  const float* sel;
  void* out;
  float* lse;
  float* w;
  int H, Hr, topk;
  int64_t nQ, nKV, nwork;
  int causal;
  float attn_scale;
  bool windows;  // stream order (StreamOrder)
};

// the LMK row's per-chunk exchange between the two waves of a pair
template <typename T>
struct LmkShared {
  T q[2][kD];       // the row's queries, by chunk parity
  T p[2][kS];       // per wave: the current slot's weighted probabilities (one per key)
  float o[2][kD];   // per wave: its slots' share of the row's output
  float lse[32];    // per slot: the row's log-sum-exp
};

// Per-lane retrieval metadata of one landmark row: lane s < K holds slot s's
// chunk index and raw score (chunk -1 for lanes >= K or rows that do not exist).
struct RowMeta {
  int j;
  float sv;
};

__device__ __forceinline__ RowMeta load_row_meta(const FwdParams& p, int64_t row_off, bool exists) {
  const int lane = threadIdx.x & 63;
  RowMeta m{-1, -INFINITY};
  if (exists && lane < p.topk) {
    m.j = p.idx[row_off + lane];
    m.sv = p.sel[row_off + lane];
  }
  return m;
}

template <typename T, bool OBO, bool XR>
__global__ __launch_bounds__(kThreads, kWgPerCu) void xattn_fwd_kernel(FwdParams p) {
  constexpr int TILE = kS * kD;
  constexpr int SQ = XR ? kS + 1 : kS;  // query rows per chunk
  static_assert(kPairs == 1, "the LMK row exchange assumes one pair per workgroup");
  __shared__ __attribute__((aligned(16))) LmkShared<T> sX[1];  // used with XR only
  __shared__ __attribute__((aligned(16))) T ring[kPairs * 2 * 2 * TILE];  // pair p: slots 2p, 2p+1 (K and V tiles)
  __shared__ int sJ[kPairs][2][32];     // [pair][chunk parity][slot]: chunk index or -1
  __shared__ int sSlot[kPairs][2][32];  // compacted lists of the valid slots: slot, chunk, weight
  __shared__ int sJc[kPairs][2][32];
  __shared__ float sWc[kPairs][2][32];
  __shared__ int sN[kPairs][2];
  // per wave, the log-sum-exp of its 32 tokens x k slots (k <= 8), stored to
  // HBM in one contiguous run at the end of the chunk instead of k scattered
  // 4-byte writes per token
  constexpr int kStageK = 8;
  __shared__ float sLse[2 * kPairs][32][kStageK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hh = lane >> 5;
  const int pair = wave >> 1, half = wave & 1;
  // Work order: workgroups are dealt to the eight XCDs round-robin (blockIdx mod
  // 8) and each wave pair is a stream of query chunks in StreamOrder (XCD ranges,
  // or chip-wide windows for long slices).
  const int xcd = (int)(blockIdx.x & 7);
  const int64_t st_wg = (int64_t)(blockIdx.x >> 3) * kPairs;
  auto order_of = [&](int q) {
    return StreamOrder((int64_t)(gridDim.x >> 3) * kPairs, st_wg + q, xcd, p.nwork, p.windows);
  };
  const StreamOrder ord = order_of(pair);
  const int64_t my_n = ord.length();
  int64_t nch = 0;  // all pairs of the workgroup run nch chunks of rounds
  for (int q = 0; q < kPairs; ++q) nch = max(nch, order_of(q).length());
  if (nch == 0) return;
  const int64_t c_begin = ord.item(0);
  const int K = p.topk;
  const int qi = 32 * half + (lane & 31);  // this lane's query token within a chunk
  const float sc = p.attn_scale * kLog2e;
  const int cb = 16 * ((lane >> 4) & 1);
  const int l32 = lane & 31;

  // work item w = (b, h, c): geometry helpers
  auto row_of = [&](const Geo& g, int64_t& row_off, bool& exists, bool& owner) __device__ {
    const int hr = p.Hr == 1 ? 0 : g.h;
    const int64_t t = p.causal ? g.c - 1 : 0;
    exists = t >= 0;
    row_off = ((g.b * p.Hr + hr) * p.nQ + (exists ? t : 0)) * K;
    owner = p.Hr != 1 || g.h == 0;  // writes the row's weights
  };
  // first wave of a pair: turn a row's metadata into the pair's compacted slot list
  auto make_slots = [&](const RowMeta& m, const Geo& g, int buf) __device__ {
    int64_t row_off;
    bool exists, owner;
    row_of(g, row_off, exists, owner);
    const bool valid = lane < K && m.j >= 0 && m.j < p.nKV;
    float mx = valid ? m.sv : -INFINITY;
    mx = max64(mx);
    const float e = valid ? expf(m.sv - mx) : 0.f;
    float sum = e;
    sum = sum64(sum);
    const float wv = valid ? e / sum : 0.f;
    const uint64_t mask = __ballot(valid);
    if (lane < 32) sJ[pair][buf][lane] = valid ? m.j : -1;
    if (valid) {
      const int rk = __popcll(mask & ((1ull << lane) - 1));
      sSlot[pair][buf][rk] = lane;
      sJc[pair][buf][rk] = m.j;
      sWc[pair][buf][rk] = wv;
    }
    if (lane == 0) sN[pair][buf] = __popcll(mask);
    if (p.w && exists && owner && lane < K) p.w[row_off + lane] = wv;
  };
  auto qrow_ptr = [&](int64_t w) __device__ {
    return reinterpret_cast<const T*>(p.q) + (w * SQ + qi) * kD;
  };
  // the LMK row's queries, copied by the first wave straight into LDS (one
  // 16-byte piece per lane below kXPieces); visible to both waves after the
  // next wait and barrier
  constexpr int kXPieces = kD * (int)sizeof(T) / 16;
  const int xh = __builtin_amdgcn_readfirstlane(half);  // the wave's half, in a scalar register
  auto load_qx = [&](int64_t w, int xbuf) __device__ {
    if (lane < kXPieces) dma_row16(reinterpret_cast<const T*>(p.q) + (w * SQ + kS) * kD, lane * 16u, &sX[0].q[xbuf][0]);
  };

  // ---- prologue: the first chunk's slot list and Q, the second chunk's metadata
  Frag<T> qf[4], qn[4];
  RowMeta meta{-1, -INFINITY};
  Geo g0(c_begin, p.nQ, p.H);  // geometry of the current chunk and of the two after it
  Geo g1 = g0, g2 = g0;  // (the range order steps without divisions)
  if (p.windows) {
    g1 = Geo(ord.item(1), p.nQ, p.H);
    g2 = Geo(ord.item(2), p.nQ, p.H);
  } else {
    g1.next(p.nQ, p.H, ord.S);
    g2 = g1;
    g2.next(p.nQ, p.H, ord.S);
  }
  if (my_n > 0) {
    int64_t ro;
    bool ex, ow;
    row_of(g0, ro, ex, ow);
    const RowMeta m0 = load_row_meta(p, ro, ex);
    const T* qr = qrow_ptr(c_begin);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) qf[kb] = load_frag(qr + 16 * kb + 8 * hh);
    if (XR && xh == 0) load_qx(c_begin, 0);
    if (half == 0) make_slots(m0, g0, 0);
    if (my_n > 1) {
      row_of(g1, ro, ex, ow);
      meta = load_row_meta(p, ro, ex);
    }
  }
  wait_vmem<0>();
  __syncthreads();

  // the pair's two ring slots alternate: cs is the slot of the next item to compute
  const TileCopy<T, 2> cp(half, lane);
  const T* const gk = reinterpret_cast<const T*>(p.k);
  const T* const gv = reinterpret_cast<const T*>(p.v);
  // element offset of the (batch, head) key/value slice of chunk w
  auto slice_of = [&](const Geo& g) __device__ { return (g.b * p.H + g.h) * p.nKV * TILE; };
  auto issue_item = [&](int64_t kvb, int j, int slot) __device__ {
    j = min(max(j, 0), (int)p.nKV - 1);  // lists hold valid chunks; never copy from outside the slice
    T* dst = ring + (2 * pair + slot) * (2 * TILE);
    cp.issue(gk + kvb + (int64_t)j * TILE, dst);
    cp.issue(gv + kvb + (int64_t)j * TILE, dst + TILE);
  };
  // lane u < 32 of the lists holds valid item u of the current chunk (slot, chunk,
  // weight); items are picked with a lane read
  int ls = sSlot[pair][0][l32], lj = sJc[pair][0][l32];
  float lw = sWc[pair][0][l32];
  int64_t kvb = uniform64(slice_of(g0)), kvb_n = 0;
  int cs = 0;
  if (my_n > 0 && sN[pair][0] > 0) issue_item(kvb, __builtin_amdgcn_readlane(lj, 0), cs);

  // bf16 fragment addresses: this lane's byte offsets inside its pair's first ring
  // slot, computed once; a round adds its slot's offset and every fragment read is
  // one of these six addresses plus an immediate (row +32, key block, V tile,
  // transposed-row gap).
  constexpr bool kB16 = std::is_same<T, __bf16>::value;
  constexpr uint32_t kTileB = TILE * sizeof(T), kRowB = kD * sizeof(T);
  const lds_char* const lds0 = (const lds_char*)(ring);
  uint32_t kofs[4], vofs[2][2];
  {
    const uint32_t pb = (uint32_t)pair * 4 * kTileB;
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

  // one retrieved chunk (item u of the current chunk, tokens from tok0) against
  // this wave's 32 queries; its tiles are in the pair's ring slot `slot`
  float ox0 = 0.f, ox1 = 0.f;  // LMK row: this lane's partial outputs for d = l%32 and 32 + l%32
  auto compute = [&](int slot, int u, int64_t tok0, int buf, f32x16& o0, f32x16& o1) __device__ {
    const uint32_t co = (uint32_t)slot * 2 * kTileB;
    const int s = __builtin_amdgcn_readlane(ls, u);
    const bool xr = XR && (u & 1) == xh;  // this wave takes the LMK row of slot u
    const T* sK = ring + (2 * pair + slot) * (2 * TILE);
    const T* sV = sK + TILE;
    // all K fragments first, so the eight products issue back to back
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
    // LMK row scores while the products run: lane l holds keys l%32 and 32 + l%32
    // over its half of the dimensions; the halves are added across l ^ 32
    float xs = 0.f;
    if (xr) {
      float a0 = 0.f, a1 = 0.f;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const Frag<T> xf = vec_frag(&sX[0].q[buf][0], 16 * kb + 8 * hh);
        a0 = frag_dot(ka[2 * kb], xf, a0);
        a1 = frag_dot(ka[2 * kb + 1], xf, a1);
      }
      a0 = sum_xor32(a0);
      a1 = sum_xor32(a1);
      xs = hh ? a1 : a0;  // the score of key `lane`
    }
    // V^T fragments are read while the softmax runs
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
    if (p.lse && hh == 0) {
      const float lv = (mx + __builtin_amdgcn_logf(sum)) * kLn2;
      if (K <= kStageK)
        sLse[wave][l32][s] = lv;
      else
        p.lse[(tok0 + qi) * K + s] = lv;
    }
    const int coef_bits = __builtin_amdgcn_readlane(__float_as_int(lw), u);
    const float coef = __int_as_float(coef_bits) * __builtin_amdgcn_rcpf(sum);
    if (xr) {
      // the LMK row's softmax over the chunk's 64 keys, one key per lane
      float xm = max64(xs) * sc;
      if (OBO) xm = fmaxf(xm, 0.f);
      const float xe = __builtin_amdgcn_exp2f(fmaf(xs, sc, -xm));
      float xsum = sum64(xe);
      if (OBO) xsum += __builtin_amdgcn_exp2f(-xm);
      if (lane == 0) sX[0].lse[s] = (xm + __builtin_amdgcn_logf(xsum)) * kLn2;
      sX[0].p[xh][lane] = (T)(xe * (__int_as_float(coef_bits) * __builtin_amdgcn_rcpf(xsum)));
    }
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
    if (xr) {
      // LMK row output: (w P) V against the V^T fragments, read again now that
      // the products have taken theirs (this wave's own probability writes are
      // read back in program order)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        __builtin_amdgcn_sched_barrier(0);  // one key block's fragments live at a time
        Frag<T> v0, v1;
        if constexpr (kB16) {
          v0 = lds_tr2(lds0 + (vofs[0][0] + co) + 16 * kb * kRowB, lds0 + (vofs[0][1] + co) + 16 * kb * kRowB);
          v1 = lds_tr2(lds0 + (vofs[1][0] + co) + 16 * kb * kRowB, lds0 + (vofs[1][1] + co) + 16 * kb * kRowB);
        } else {
          v0 = lds_frag_t(sV, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, cb);
          v1 = lds_frag_t(sV, 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh, 32 + cb);
        }
        const Frag<T> xf = vec_frag_t(&sX[0].p[xh][0], 16 * kb + 4 * hh, 16 * kb + 8 + 4 * hh);
        ox0 = frag_dot(v0, xf, ox0);
        ox1 = frag_dot(v1, xf, ox1);
      }
    }
  };

  // Every chunk takes K rounds (a pair whose chunk has fewer valid slots, or that
  // has run out of chunks, idles), so both pairs meet the same barriers.  Each
  // round: wait for this wave's copies, barrier (the partner's copies are visible
  // and the slot read last round is free), copy the pair's next item into that
  // slot, then compute this round's item.
  f32x16 o0 = zero16(), o1 = zero16();
  for (int64_t ci = 0; ci < nch; ++ci) {
    const bool live = ci < my_n, live_next = ci + 1 < my_n;
    const int buf = (int)(ci & 1);
    const int n = live ? sN[pair][buf] : 0;
    const int64_t w = ord.item(ci), w_next = ord.item(ci + 1);
    const int64_t tok0 = w * SQ;
    for (int u = 0; u < K; ++u) {
      wait_vmem<0>();
      block_barrier();
      if (u == 0) {
        if (!XR && ci > 0 && live) {
#pragma unroll
          for (int kb = 0; kb < 4; ++kb) qf[kb] = qn[kb];
        }
        if (ci > 0 && live) {
          ls = sSlot[pair][buf][l32];
          lj = sJc[pair][buf][l32];
          lw = sWc[pair][buf][l32];
          kvb = kvb_n;
        }
        if (live_next) {
          if constexpr (!XR) {
            const T* qr = qrow_ptr(w_next);
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) qn[kb] = load_frag(qr + 16 * kb + 8 * hh);
          } else if (xh == 0) {
            load_qx(w_next, buf ^ 1);
          }
          if (half == 0) make_slots(meta, g1, buf ^ 1);
          if (ci + 2 < my_n) {
            int64_t ro;
            bool ex, ow;
            row_of(g2, ro, ex, ow);
            meta = load_row_meta(p, ro, ex);
          }
          kvb_n = uniform64(slice_of(g1));
        }
        if (K == 1) block_barrier();  // the next chunk's list is needed this round
      }
      const bool comp = u < n;
      const int is = comp ? cs ^ 1 : cs;
      if (u + 1 < n) {
        issue_item(kvb, __builtin_amdgcn_readlane(lj, u + 1), is);
      } else if (u == K - 1 && live_next && sN[pair][buf ^ 1] > 0) {
        issue_item(kvb_n, sJc[pair][buf ^ 1][0], is);
      }
      if (comp) {
        compute(cs, u, tok0, buf, o0, o1);
        cs ^= 1;
      }
    }
    // with the LMK row the next chunk's Q rows are loaded only now, straight into
    // the fragments (the registers of a prefetch are what the row's own work
    // needs); the next round's wait covers them
    if (XR && live_next) {
      const T* qr = qrow_ptr(w_next);
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) qf[kb] = load_frag(qr + 16 * kb + 8 * hh);
    }

    // ---- finish the chunk: each wave stores its 32 query rows
    if (live) {
      T* orow = reinterpret_cast<T*>(p.out) + (tok0 + qi) * kD;
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        store4(orow + 8 * gq + 4 * hh, o0[4 * gq], o0[4 * gq + 1], o0[4 * gq + 2], o0[4 * gq + 3]);
        store4(orow + 32 + 8 * gq + 4 * hh, o1[4 * gq], o1[4 * gq + 1], o1[4 * gq + 2], o1[4 * gq + 3]);
      }
      if (p.lse && K <= kStageK) {
        // this wave's tokens are one contiguous run of 32 k entries; slots
        // without a chunk read -inf
        const int64_t base = (tok0 + 32 * half) * K;
        for (int e = lane; e < 32 * K; e += 64) {
          const int tk = e / K, sl = e - tk * K;
          p.lse[base + e] = sJ[pair][buf][sl] < 0 ? -INFINITY : sLse[wave][tk][sl];
        }
      } else if (p.lse && n < K && hh == 0) {
        float* lse = p.lse + (tok0 + qi) * K;
        for (int s = 0; s < K; ++s)
          if (sJ[pair][buf][s] < 0) lse[s] = -INFINITY;
      }
      if constexpr (XR) {
        // the LMK row: add the two waves' shares (each lane first adds its key
        // half to the partner lane's), then one wave stores the row and its lse
        const float t0 = sum_xor32(ox0), t1 = sum_xor32(ox1);
        sX[0].o[xh][lane] = hh ? t1 : t0;  // lane l: d = l
        block_barrier();
        if (xh == 0) {
          const int64_t tx = tok0 + kS;
          reinterpret_cast<T*>(p.out)[tx * kD + lane] = (T)(sX[0].o[0][lane] + sX[0].o[1][lane]);
          if (p.lse && lane < K) p.lse[tx * K + lane] = sJ[pair][buf][lane] < 0 ? -INFINITY : sX[0].lse[lane];
        }
        ox0 = 0.f;
        ox1 = 0.f;
      }
      // the causal last row feeds no chunk: its weights go out with chunk 0
      if (p.w && p.causal && g0.c == 0 && half == 1) {
        int64_t ro;
        bool ex, ow;
        row_of(g0, ro, ex, ow);
        if (ow) {
          const int64_t last_off = (g0.b * p.Hr + (p.Hr == 1 ? 0 : g0.h)) * p.nQ * K + (p.nQ - 1) * K;
          float wv;
          int jv;
          wave_row_weight(p.idx, p.sel, last_off, K, p.nKV, wv, jv);
          if (lane < K) p.w[last_off + lane] = wv;
        }
      }
    }
    o0 = zero16();
    o1 = zero16();
    g0 = g1;
    g1 = g2;
    if (p.windows)
      g2 = Geo(ord.item(ci + 3), p.nQ, p.H);
    else
      g2.next(p.nQ, p.H, ord.S);
  }
}

}  // namespace

hipError_t launch_xattn_fwd(const Shape& s, const void* q, const void* k, const void* v,
                            const int32_t* idx, const float* sel, void* out, float* lse, float* w,
                            hipStream_t stream) {
  if (!s.causal) return launch_xattn_decode(s, nullptr, nullptr, q, k, v, const_cast<int32_t*>(idx),
                                            const_cast<float*>(sel), out, lse, w, nullptr, nullptr, stream);
  FwdParams p;
  p.q = q; p.k = k; p.v = v; p.idx = idx; p.sel = sel;
  p.out = out; p.lse = lse; p.w = w;
  p.H = s.H; p.Hr = s.Hr; p.topk = s.topk;
  p.nQ = s.nQ; p.nKV = s.nKV;
  p.nwork = (int64_t)s.B * s.H * s.nQ;
  p.causal = s.causal;
  p.attn_scale = s.attn_scale;
  p.windows = use_window_order(s.nKV, s.bf16 ? 2 : 4);
  const bool xr = s.Sq != kS;
  // persistent workgroups: kWgPerCu per CU, a multiple of 8 (one share per XCD),
  // each running kPairs chunk streams
  const int64_t target = round8((int64_t)device_cus() * kWgPerCu), wgs = (p.nwork + kPairs - 1) / kPairs;
  const dim3 grid((unsigned)(wgs < target ? round8(wgs) : target)), block(kThreads);
  auto go = [&](auto kernel) { launch_kernel("xattn_fwd_kernel", kernel, grid, block, 0, stream, p); };
  if (s.bf16) {
    if (xr) s.off_by_one ? go(xattn_fwd_kernel<__bf16, true, true>) : go(xattn_fwd_kernel<__bf16, false, true>);
    else s.off_by_one ? go(xattn_fwd_kernel<__bf16, true, false>) : go(xattn_fwd_kernel<__bf16, false, false>);
  } else {
    if (xr) s.off_by_one ? go(xattn_fwd_kernel<float, true, true>) : go(xattn_fwd_kernel<float, false, true>);
    else s.off_by_one ? go(xattn_fwd_kernel<float, true, false>) : go(xattn_fwd_kernel<float, false, false>);
  }
  return take_launch_error();
}

}  // namespace gca
