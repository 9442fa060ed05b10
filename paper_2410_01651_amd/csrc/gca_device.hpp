// Device-side building blocks for the GCA kernels (gfx950 / CDNA4, wave64).
//
// Matrix products use the 32x32 MFMA tiles with fp32 accumulation.  A
// "fragment" is what one lane feeds one 32x32x16 step: 8 consecutive entries
// of the contraction dimension.  For an A operand (rows x k) lane l holds row
// l%32 and k = 8*(l/32) + 0..7; for a B operand (k x cols) lane l holds column
// l%32 and the same k range.  The 32x32 accumulator gives lane l column l%32
// and rows 8*(i/4) + 4*(l/32) + i%4 for register i = 0..15.
//
// bf16 fragments feed one v_mfma_f32_32x32x16_bf16; fp32 fragments feed eight
// v_mfma_f32_32x32x2f32 (step m takes entry m of every lane, so the eight
// steps together contract the same 16 k-entries).  Either way the operand and
// accumulator layouts are identical, so every kernel is written once for both.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gca {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4_tr;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

constexpr int kS = 64;        // tokens per chunk
constexpr int kD = 64;        // head dimension
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

struct f32x8 {
  f32x4 lo, hi;
};

template <typename T> struct FragOf;
template <> struct FragOf<__bf16> { using type = bf16x8; };
template <> struct FragOf<float> { using type = f32x8; };
template <typename T> using Frag = typename FragOf<T>::type;

// ---------------------------------------------------------------- MFMA ----

__device__ __forceinline__ void mma32(f32x16& c, const bf16x8& a, const bf16x8& b) {
  c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ void mma32(f32x16& c, const f32x8& a, const f32x8& b) {
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.lo[0], b.lo[0], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.lo[1], b.lo[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.lo[2], b.lo[2], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.lo[3], b.lo[3], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.hi[0], b.hi[0], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.hi[1], b.hi[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.hi[2], b.hi[2], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.hi[3], b.hi[3], c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

// ------------------------------------------------------- fragment loads ----

// 8 consecutive elements starting at p (row-major operand, k contiguous).
__device__ __forceinline__ bf16x8 load_frag(const __bf16* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}
__device__ __forceinline__ f32x8 load_frag(const float* p) {
  f32x8 f;
  f.lo = *reinterpret_cast<const f32x4*>(p);
  f.hi = *reinterpret_cast<const f32x4*>(p + 4);
  return f;
}

__device__ __forceinline__ bf16x8 zero_frag(const __bf16*) {
  bf16x8 z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = (__bf16)0.f;
  return z;
}
__device__ __forceinline__ f32x8 zero_frag(const float*) {
  f32x8 z;
  z.lo = f32x4{0.f, 0.f, 0.f, 0.f};
  z.hi = z.lo;
  return z;
}

// Fragment whose contraction runs down a column of a row-major LDS tile M
// (leading dimension ld): lane l gets M[r0 + e][col] for e = 0..3 followed by
// M[r1 + e][col], where col = cbase + l%16 and cbase is the column base of the
// lane's 16-lane group.  For bf16 this is two ds_read_b64_tr_b16: within a
// 16-lane group, source lane s reads 4 elements of row r + s/4 at column
// cbase + 4*(s%4), and the hardware hands lane i element i%4 of source lane
// 4e + i/4, i.e. M[r + e][cbase + i].
__device__ __forceinline__ bf16x8 load_frag_t(const __bf16* M, int ld, int r0, int r1, int cbase) {
  const int s = threadIdx.x & 15;
  const __bf16* p0 = M + (r0 + (s >> 2)) * ld + cbase + 4 * (s & 3);
  const __bf16* p1 = M + (r1 + (s >> 2)) * ld + cbase + 4 * (s & 3);
  typedef __attribute__((address_space(3))) bf16x4_tr lds_v4;
  bf16x4_tr a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_v4*)(p0));
  bf16x4_tr b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_v4*)(p1));
  bf16x8 f;
  f[0] = a[0]; f[1] = a[1]; f[2] = a[2]; f[3] = a[3];
  f[4] = b[0]; f[5] = b[1]; f[6] = b[2]; f[7] = b[3];
  return f;
}
__device__ __forceinline__ f32x8 load_frag_t(const float* M, int ld, int r0, int r1, int cbase) {
  const int col = cbase + (threadIdx.x & 15);
  f32x8 f;
  f.lo = f32x4{M[(r0 + 0) * ld + col], M[(r0 + 1) * ld + col], M[(r0 + 2) * ld + col],
               M[(r0 + 3) * ld + col]};
  f.hi = f32x4{M[(r1 + 0) * ld + col], M[(r1 + 1) * ld + col], M[(r1 + 2) * ld + col],
               M[(r1 + 3) * ld + col]};
  return f;
}

// Build a B/A fragment from accumulator registers: entries 8*half .. 8*half+7
// of a 32x32 accumulator, scaled.  Used to feed a softmax tile held in the
// accumulator layout back into the next product without leaving registers.
__device__ __forceinline__ void frag_from_acc(bf16x8& f, const f32x16& acc, int half, float scale) {
#pragma unroll
  for (int m = 0; m < 8; ++m) f[m] = (__bf16)(acc[8 * half + m] * scale);
}
__device__ __forceinline__ void frag_from_acc(f32x8& f, const f32x16& acc, int half, float scale) {
  f.lo = f32x4{acc[8 * half + 0], acc[8 * half + 1], acc[8 * half + 2], acc[8 * half + 3]} * scale;
  f.hi = f32x4{acc[8 * half + 4], acc[8 * half + 5], acc[8 * half + 6], acc[8 * half + 7]} * scale;
}

// ------------------------------------------------------- element stores ----

// Store 4 consecutive fp32 values as the tensor dtype.
__device__ __forceinline__ void store4(__bf16* p, float a, float b, float c, float d) {
  typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 v4;
  v4 v;
  v[0] = (__bf16)a; v[1] = (__bf16)b; v[2] = (__bf16)c; v[3] = (__bf16)d;
  *reinterpret_cast<v4*>(p) = v;
}
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<f32x4*>(p) = f32x4{a, b, c, d};
}

__device__ __forceinline__ float to_f32(__bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f32(float x) { return x; }

// 16-byte global <-> LDS staging of a 64 x 64 tile (row-major source, leading
// dimension 64) into an LDS tile with leading dimension ld, by nthreads threads.
template <typename T, int NTHREADS>
struct Tile64 {
  static constexpr int kVec = 16 / sizeof(T);               // elements per 16 bytes
  static constexpr int kPerThread = kS * kD / kVec / NTHREADS;
  u32x4 r[kPerThread];

  __device__ __forceinline__ void load(const T* __restrict__ src, int tid) {
#pragma unroll
    for (int it = 0; it < kPerThread; ++it) {
      const int u = tid + NTHREADS * it;
      const int row = u / (kD / kVec), col = (u % (kD / kVec)) * kVec;
      r[it] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + row * kD + col));
    }
  }
  __device__ __forceinline__ void load_cached(const T* __restrict__ src, int tid) {
#pragma unroll
    for (int it = 0; it < kPerThread; ++it) {
      const int u = tid + NTHREADS * it;
      const int row = u / (kD / kVec), col = (u % (kD / kVec)) * kVec;
      r[it] = *reinterpret_cast<const u32x4*>(src + row * kD + col);
    }
  }
  __device__ __forceinline__ void store(T* dst, int ld, int tid) const {
#pragma unroll
    for (int it = 0; it < kPerThread; ++it) {
      const int u = tid + NTHREADS * it;
      const int row = u / (kD / kVec), col = (u % (kD / kVec)) * kVec;
      *reinterpret_cast<u32x4*>(dst + row * ld + col) = r[it];
    }
  }
};

// ------------------------------------------------------ cross-lane ops ----

__device__ __forceinline__ float xor32(float x) { return __shfl_xor(x, 32); }

// Map a 1-D block id to a logical work id so that each of the 8 XCDs (which
// receive blocks round-robin) works on one contiguous range of logical ids and
// its private L2 sees a coherent working set.  The grid must be a multiple of 8
// blocks; ids >= n are padding and must exit.
__device__ __forceinline__ int64_t xcd_swizzle(int64_t bid, int64_t grid) {
  const int64_t per = grid >> 3;
  return (bid & 7) * per + (bid >> 3);
}

// ---------------------------------------------------- top-k selection ----

// Ordering of retrieval candidates: higher score first, ties to lower chunk index.
__device__ __forceinline__ bool better(float s, int j, float s2, int j2) {
  return s > s2 || (s == s2 && j < j2);
}

constexpr int kNoChunk = 0x7fffffff;

// A lane's running best-KM list, sorted best first, in registers.
template <int KM>
struct TopList {
  float s[KM];
  int j[KM];

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int i = 0; i < KM; ++i) { s[i] = -INFINITY; j[i] = kNoChunk; }
  }
  // Insert (cs, cj) if it beats the current last entry.
  __device__ __forceinline__ void insert(float cs, int cj) {
    if (!better(cs, cj, s[KM - 1], j[KM - 1])) return;
#pragma unroll
    for (int i = KM - 1; i > 0; --i) {
      const bool above = better(cs, cj, s[i - 1], j[i - 1]);
      const bool here = better(cs, cj, s[i], j[i]);
      const float ns = above ? s[i - 1] : (here ? cs : s[i]);
      const int nj = above ? j[i - 1] : (here ? cj : j[i]);
      s[i] = ns; j[i] = nj;
    }
    if (better(cs, cj, s[0], j[0])) { s[0] = cs; j[0] = cj; }
  }
  __device__ __forceinline__ void pop() {
#pragma unroll
    for (int i = 0; i < KM - 1; ++i) { s[i] = s[i + 1]; j[i] = j[i + 1]; }
    s[KM - 1] = -INFINITY; j[KM - 1] = kNoChunk;
  }
};

// Wave-wide best of one (score, chunk) per lane.
__device__ __forceinline__ void wave_best(float& s, int& j) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float os = __shfl_xor(s, off);
    const int oj = __shfl_xor(j, off);
    if (better(os, oj, s, j)) { s = os; j = oj; }
  }
}

// Merge the 64 lanes' lists into the wave's best k (k <= 64).  Lane r < *count
// receives the r-th best (score, chunk); *count <= k is the number of real
// candidates.  Lists are consumed.
template <int KM>
__device__ __forceinline__ void wave_merge(TopList<KM>& L, int k, float& my_s, int& my_j, int& count) {
  const int lane = threadIdx.x & 63;
  my_s = -INFINITY;
  my_j = kNoChunk;
  count = 0;
  for (int r = 0; r < k; ++r) {
    float bs = L.s[0];
    int bj = L.j[0];
    wave_best(bs, bj);
    if (bj == kNoChunk) break;
    if (L.j[0] == bj) L.pop();
    if (lane == r) { my_s = bs; my_j = bj; }
    ++count;
  }
}

// Position of lane r's chunk among the first `count` lanes' chunks in
// ascending chunk order (chunks are distinct).
__device__ __forceinline__ int rank_by_chunk(int my_j, int count) {
  int rank = 0;
  for (int r = 0; r < count; ++r) {
    const int oj = __shfl(my_j, r);
    rank += (oj < my_j) ? 1 : 0;
  }
  return rank;
}

// Fusion weight (Eq. 2) of slot s of one retrieval row: softmax over the valid
// slots (0 <= idx < nKV) of the raw retrieval scores; 0 and chunk -1 for pads.
__device__ __forceinline__ void row_weight(const int32_t* __restrict__ idx_row, const float* __restrict__ sel_row,
                               int K, int64_t nKV, int s, float& w, int& j) {
  float m = -INFINITY;
  for (int u = 0; u < K; ++u) {
    const int ju = idx_row[u];
    if (ju >= 0 && ju < nKV) m = fmaxf(m, sel_row[u]);
  }
  float sum = 0.f;
  for (int u = 0; u < K; ++u) {
    const int ju = idx_row[u];
    if (ju >= 0 && ju < nKV) sum += expf(sel_row[u] - m);
  }
  const int js = idx_row[s];
  const bool valid = js >= 0 && js < nKV;
  w = valid ? expf(sel_row[s] - m) / sum : 0.f;
  j = valid ? js : -1;
}

}  // namespace gca
