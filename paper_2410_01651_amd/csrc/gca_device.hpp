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

#include <type_traits>

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

// x, as a value the compiler cannot prove loop-invariant: an address formed
// from it is computed where it is used instead of being hoisted and held in
// registers across a loop (for kernels at the edge of their register budget).
__device__ __forceinline__ int opaque(int x) {
  __asm__ volatile("" : "+v"(x));
  return x;
}

// Number of set bits of a wave-wide mask below this lane (v_mbcnt: no lane mask
// is formed or kept in registers).
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
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

// Entry m of a fragment as fp32.  For bf16 this reads the packed bits (one shift
// or mask), so the compiler cannot re-derive the value by converting the fp32
// source again (two instructions per entry).
__device__ __forceinline__ float frag_elem(const bf16x8& f, int m) {
  const u32x4 w = __builtin_bit_cast(u32x4, f);
  const uint32_t x = w[m >> 1];
  return __uint_as_float((m & 1) ? (x & 0xffff0000u) : (x << 16));
}
__device__ __forceinline__ float frag_elem(const f32x8& f, int m) { return m < 4 ? f.lo[m] : f.hi[m - 4]; }

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

// ------------------------------------------- asynchronous tile staging ----
//
// Chunk tiles (64 tokens x 64 dims, row-major in HBM) are copied straight into
// LDS with global_load_lds_dwordx4: each lane supplies a global address and the
// 64 lanes of one instruction fill 1 KB of consecutive LDS.  The LDS copy is
// XOR-swizzled at 16-byte granularity: LDS chunk c' of row r holds the row's
// global chunk c' ^ sw(r).  The LDS serves 256 bytes (64 banks) per cycle: a
// 16-byte read per lane (A/B fragments, lane l on row l mod 32) takes 16 lanes
// per cycle, i.e. 16 consecutive rows, and a bf16 row is 128 bytes, so the 8
// rows of one parity among them share a bank window and must take 8 different
// chunks; the transposed 8-byte reads (32 lanes per cycle: rows r0 .. r0 + 3,
// each four adjacent chunks 4 m .. 4 m + 3) need rows r0 and r0 + 2 (one
// window) in different halves of the row.  For bf16, sw(r) = (b0 ^ b3) +
// 2 b2 + 4 b1 (bits b of r mod 16) does both, and also keeps any 8 aligned
// consecutive rows apart; it repeats every 16 rows, so row offsets of +16 and +32
// stay constant displacements but +8 does not (the transposed reads at +8 rows
// take their own addresses).  An fp32 row is 256 bytes (16 chunks): sw(r) =
// r mod 16 already spreads 16 consecutive rows over the banks.
//
// The copies are asynchronous: a wave's own copies are complete once its
// vector-memory counter has dropped to the number issued after them
// (wait_vmem), and the other waves' copies once all waves have passed the next
// barrier (block_barrier).  block_barrier deliberately does not drain the
// counter, so copies for later slots stay in flight across it; no global store
// or load into registers may be issued between a copy and the wait for it.

template <typename T>
struct Swz {
  static constexpr int kVec = 16 / sizeof(T);  // elements per 16-byte chunk
  static constexpr int kCPR = kD / kVec;       // chunks per row (8 bf16, 16 fp32)
  __device__ static __forceinline__ int sw(int r) {
    if constexpr (kCPR == 8) return ((r ^ (r >> 3)) & 1) | ((r >> 1) & 2) | ((r << 1) & 4);
    else return r & (kCPR - 1);
  }
  __device__ static __forceinline__ int off(int r, int col) {
    return r * kD + (((col / kVec) ^ sw(r)) * kVec) + (col % kVec);
  }
};

template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier that leaves vector-memory operations (the asynchronous tile
// copies) in flight: it first drains this wave's LDS operations, so that LDS
// written before the barrier is visible to every wave after it (s_barrier alone
// does not wait for a wave's outstanding LDS writes).
__device__ __forceinline__ void block_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// A wave-uniform global address in scalar registers (the read-back builtin returns
// a signed int: each half is widened through uint32_t, never sign-extended).
__device__ __forceinline__ uint64_t uniform_addr(const void* g) {
  const uint64_t ga = (uint64_t)(uintptr_t)g;
  return (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)ga) |
         ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(ga >> 32)) << 32);
}
// A wave-uniform 64-bit integer forced into scalar registers.
__device__ __forceinline__ int64_t uniform64(int64_t x) {
  return (int64_t)((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)x) |
                   ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32)) << 32));
}
// A wave-uniform LDS byte address (plus a wave-uniform offset) in a scalar register.
__device__ __forceinline__ uint32_t uniform_lds(const void* lds, uint32_t add = 0) {
  return __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) char*)lds) + add);
}

// The same tile copy with this lane's global byte offsets computed once.  A copy
// then takes the tile's global base in scalar registers and a 32-bit lane offset
// (the scalar-base form of the instruction), so issuing a tile costs one scalar
// move and one vector-memory instruction per 16-byte chunk and no vector address
// arithmetic.  `g` and `lds` must hold the same value in every lane.
// ROWS: rows of the tile (64, or 32 for a half tile).
template <typename T, int NW, int ROWS = kS>
struct TileCopy {
  static constexpr int kVec = Swz<T>::kVec, kCPR = Swz<T>::kCPR, kN = kCPR * ROWS / (64 * NW);
  static_assert(kN >= 1 && kN * 64 * NW == kCPR * ROWS, "the waves' 16-byte pieces cover the tile");
  uint32_t goff[kN];
  uint32_t lwave;  // this wave's first 1 KiB block of the tile in LDS (scalar)

  // row_stride: elements between consecutive source rows (kD: a contiguous tile);
  // rows: source rows that exist (LDS rows past them repeat the last one)
  __device__ __forceinline__ TileCopy(int wave, int lane, int row_stride = kD, int rows = kS) {
#pragma unroll
    for (int ii = 0; ii < kN; ++ii) {
      const int pch = (ii * NW + wave) * 64 + lane;
      const int r = pch / kCPR;
      const int c = (pch % kCPR) ^ Swz<T>::sw(r);
      const int rs = r < rows ? r : rows - 1;
      goff[ii] = (uint32_t)((rs * row_stride + c * kVec) * sizeof(T));
    }
    lwave = __builtin_amdgcn_readfirstlane((uint32_t)(wave * 64 * 16));
  }
  __device__ __forceinline__ void issue(const T* g, const T* lds) const {
    const uint64_t gs = uniform_addr(g);
    const uint32_t lb = uniform_lds(lds) + lwave;
#pragma unroll
    for (int ii = 0; ii < kN; ++ii)
      asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(goff[ii]), "s"(gs),
                   "s"(lb + ii * NW * 64 * 16)
                   : "m0");
  }
};

// The active lanes of a wave each copy 16 bytes at g + lane_off into LDS at
// lds + 16 * lane (one row of a tile: lane_off = 16 * lane); g and lds
// wave-uniform.
__device__ __forceinline__ void dma_row16(const void* g, uint32_t lane_off, const void* lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(lane_off), "s"(uniform_addr(g)),
               "s"(uniform_lds(lds))
               : "m0");
}

// One wave copies 64 floats at g + lane_off (bytes, lane_off = lane * stride
// precomputed) into 64 consecutive LDS floats; g and lds wave-uniform.
__device__ __forceinline__ void dma_column_s(const float* g, uint32_t lane_off, const float* lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1" ::"v"(lane_off), "s"(uniform_addr(g)),
               "s"(uniform_lds(lds))
               : "m0");
}

// Fragments from a swizzled tile: 8 consecutive elements of row r from column col
// (a multiple of 8) ...
__device__ __forceinline__ bf16x8 lds_frag(const __bf16* tile, int r, int col) {
  return *reinterpret_cast<const bf16x8*>(tile + Swz<__bf16>::off(r, col));
}
__device__ __forceinline__ f32x8 lds_frag(const float* tile, int r, int col) {
  f32x8 f;
  f.lo = *reinterpret_cast<const f32x4*>(tile + Swz<float>::off(r, col));
  f.hi = *reinterpret_cast<const f32x4*>(tile + Swz<float>::off(r, col + 4));
  return f;
}
// Fragment reads at precomputed LDS byte addresses (address space 3), so that a
// constant displacement folds into the instruction's offset field.
typedef __attribute__((address_space(3))) char lds_char;
__device__ __forceinline__ bf16x8 lds_b128_at(const lds_char* p) {
  return *reinterpret_cast<const __attribute__((address_space(3))) bf16x8*>(p);
}
// Transposed fragment (see lds_frag_t): the two 8-byte transposed reads at p0
// and p1 (rows r0.. and r1.. of the same 16 columns).
__device__ __forceinline__ bf16x8 lds_tr2(const lds_char* p0, const lds_char* p1) {
  typedef __attribute__((address_space(3))) bf16x4_tr lds_v4;
  bf16x4_tr a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_v4*)(p0));
  bf16x4_tr b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_v4*)(p1));
  bf16x8 f;
  f[0] = a[0]; f[1] = a[1]; f[2] = a[2]; f[3] = a[3];
  f[4] = b[0]; f[5] = b[1]; f[6] = b[2]; f[7] = b[3];
  return f;
}

// Fragment whose contraction runs down a column of a row-major swizzled LDS
// tile M: lane l gets M[r0 + e][col] for e = 0..3 followed by M[r1 + e][col],
// where col = cbase + l%16 and cbase is the column base of the lane's 16-lane
// group.  For bf16 this is two ds_read_b64_tr_b16: within a
// 16-lane group, source lane s reads 4 elements of row r + s/4 at column
// cbase + 4*(s%4), and the hardware hands lane i element i%4 of source lane
// 4e + i/4, i.e. M[r + e][cbase + i].
__device__ __forceinline__ bf16x8 lds_frag_t(const __bf16* tile, int r0, int r1, int cbase) {
  const int s = threadIdx.x & 15;
  typedef __attribute__((address_space(3))) bf16x4_tr lds_v4;
  const __bf16* p0 = tile + Swz<__bf16>::off(r0 + (s >> 2), cbase + 4 * (s & 3));
  const __bf16* p1 = tile + Swz<__bf16>::off(r1 + (s >> 2), cbase + 4 * (s & 3));
  bf16x4_tr a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_v4*)(p0));
  bf16x4_tr b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_v4*)(p1));
  bf16x8 f;
  f[0] = a[0]; f[1] = a[1]; f[2] = a[2]; f[3] = a[3];
  f[4] = b[0]; f[5] = b[1]; f[6] = b[2]; f[7] = b[3];
  return f;
}
__device__ __forceinline__ f32x8 lds_frag_t(const float* tile, int r0, int r1, int cbase) {
  const int col = cbase + (threadIdx.x & 15);
  using Z = Swz<float>;
  f32x8 f;
  f.lo = f32x4{tile[Z::off(r0, col)], tile[Z::off(r0 + 1, col)], tile[Z::off(r0 + 2, col)],
               tile[Z::off(r0 + 3, col)]};
  f.hi = f32x4{tile[Z::off(r1, col)], tile[Z::off(r1 + 1, col)], tile[Z::off(r1 + 2, col)],
               tile[Z::off(r1 + 3, col)]};
  return f;
}

// ------------------------------------------- one row against a tile ----
//
// A single query row (the LMK row of a chunk) against a tile whose fragments a
// wave already holds: the row is a plain vector x[64] in LDS, read in the entry
// order of the fragment it meets, and the products run on the VALU as fp32 dot
// products (v_dot2_f32_bf16 for bf16: exact products, fp32 sums, as on MFMA).

// sum_m a[m] b[m] + acc over the 8 entries of two fragments
__device__ __forceinline__ float frag_dot(const bf16x8& a, const bf16x8& b, float acc) {
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 0, 1), __builtin_shufflevector(b, b, 0, 1),
                                        acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 2, 3), __builtin_shufflevector(b, b, 2, 3),
                                        acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 4, 5), __builtin_shufflevector(b, b, 4, 5),
                                        acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 6, 7), __builtin_shufflevector(b, b, 6, 7),
                                        acc, false);
  return acc;
}
__device__ __forceinline__ float frag_dot(const f32x8& a, const f32x8& b, float acc) {
#pragma unroll
  for (int m = 0; m < 4; ++m) acc = fmaf(a.lo[m], b.lo[m], acc);
#pragma unroll
  for (int m = 0; m < 4; ++m) acc = fmaf(a.hi[m], b.hi[m], acc);
  return acc;
}
// A fragment whose entry 0 is x and whose other entries are 0.
template <typename T> __device__ __forceinline__ Frag<T> frag_e0(float x);
template <> __device__ __forceinline__ bf16x8 frag_e0<__bf16>(float x) {
  bf16x8 f;
#pragma unroll
  for (int m = 0; m < 8; ++m) f[m] = (__bf16)0.f;
  f[0] = (__bf16)x;
  return f;
}
template <> __device__ __forceinline__ f32x8 frag_e0<float>(float x) {
  f32x8 f;
  f.lo = f32x4{x, 0.f, 0.f, 0.f};
  f.hi = f32x4{0.f, 0.f, 0.f, 0.f};
  return f;
}
template <typename T> __device__ __forceinline__ Frag<T> zero_frag();
template <> __device__ __forceinline__ bf16x8 zero_frag<__bf16>() { return frag_e0<__bf16>(0.f); }
template <> __device__ __forceinline__ f32x8 zero_frag<float>() { return frag_e0<float>(0.f); }
// Entries 0 .. n-1 of f kept, the rest set to 0.
template <typename T> __device__ __forceinline__ Frag<T> frag_prefix(Frag<T> f, int n);
template <> __device__ __forceinline__ bf16x8 frag_prefix<__bf16>(bf16x8 f, int n) {
#pragma unroll
  for (int m = 0; m < 8; ++m)
    if (m >= n) f[m] = (__bf16)0.f;
  return f;
}
template <> __device__ __forceinline__ f32x8 frag_prefix<float>(f32x8 f, int n) {
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    if (m >= n) f.lo[m] = 0.f;
    if (m + 4 >= n) f.hi[m] = 0.f;
  }
  return f;
}
// Entries x[c .. c+7]: meets a row fragment (contraction along the row).
template <typename T>
__device__ __forceinline__ Frag<T> vec_frag(const T* x, int c) {
  return load_frag(x + c);
}
// Entries x[r0 .. r0+3] then x[r1 .. r1+3]: meets a column fragment (lds_frag_t,
// lds_tr2) or the probability fragments built from an accumulator.
__device__ __forceinline__ bf16x8 vec_frag_t(const __bf16* x, int r0, int r1) {
  typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 v4;
  const v4 a = *reinterpret_cast<const v4*>(x + r0), b = *reinterpret_cast<const v4*>(x + r1);
  bf16x8 f;
  f[0] = a[0]; f[1] = a[1]; f[2] = a[2]; f[3] = a[3];
  f[4] = b[0]; f[5] = b[1]; f[6] = b[2]; f[7] = b[3];
  return f;
}
__device__ __forceinline__ f32x8 vec_frag_t(const float* x, int r0, int r1) {
  f32x8 f;
  f.lo = *reinterpret_cast<const f32x4*>(x + r0);
  f.hi = *reinterpret_cast<const f32x4*>(x + r1);
  return f;
}

// ------------------------------------------------------ cross-lane ops ----

// ------------------------------------------------ cross-lane exchange ----
//
// Butterfly reductions without the LDS crossbar (ds_bpermute costs a round trip
// per step): DPP quad permutes swap lanes l ^ 1 and l ^ 2, DPP row rotations by
// 4 and 8 reach the other quads of a 16-lane row (the half-row mirror the other
// quad of an 8-lane group), and v_permlane16_swap /
// v_permlane32_swap hand every lane the pair {x[l], x[l ^ 16]} / {x[l], x[l ^ 32]}.
constexpr int kDppXor1 = 0xB1;   // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;   // quad_perm [2, 3, 0, 1]
constexpr int kDppRor4 = 0x124;  // row_ror:4
constexpr int kDppRor8 = 0x128;  // row_ror:8
constexpr int kDppHalfMirror = 0x141;  // row_half_mirror: lane i of 8 <-> lane 7 - i

template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __uint_as_float(dpp<CTRL>(__float_as_uint(x)));
}
template <int CTRL>
__device__ __forceinline__ int dpp(int x) {
  return (int)dpp<CTRL>((uint32_t)x);
}
// {x[l], x[l ^ 16]} and {x[l], x[l ^ 32]} (in either order)
__device__ __forceinline__ void pair16(uint32_t x, uint32_t& a, uint32_t& b) {
  const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  a = r[0];
  b = r[1];
}
__device__ __forceinline__ void pair32(uint32_t x, uint32_t& a, uint32_t& b) {
  const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  a = r[0];
  b = r[1];
}

// Sum over each 32-lane half (every lane of the half gets it).
__device__ __forceinline__ float sum32(float x) {
  x += dpp<kDppXor1>(x);
  x += dpp<kDppXor2>(x);
  x += dpp<kDppRor4>(x);
  x += dpp<kDppRor8>(x);
  uint32_t a, b;
  pair16(__float_as_uint(x), a, b);
  return __uint_as_float(a) + __uint_as_float(b);
}
// Maximum of the 32 entries of two accumulators, as a tree of three-operand
// maxima (v_max3_f32: 16 instructions for 32 values).
__device__ __forceinline__ float max_of(const f32x16& a, const f32x16& b) {
  float m[11];
#pragma unroll
  for (int i = 0; i < 5; ++i) m[i] = fmaxf(fmaxf(a[3 * i], a[3 * i + 1]), a[3 * i + 2]);
#pragma unroll
  for (int i = 0; i < 5; ++i) m[5 + i] = fmaxf(fmaxf(b[3 * i], b[3 * i + 1]), b[3 * i + 2]);
  m[10] = fmaxf(a[15], b[15]);
  const float x0 = fmaxf(fmaxf(m[0], m[1]), m[2]), x1 = fmaxf(fmaxf(m[3], m[4]), m[5]);
  const float x2 = fmaxf(fmaxf(m[6], m[7]), m[8]), x3 = fmaxf(m[9], m[10]);
  return fmaxf(fmaxf(x0, x1), fmaxf(x2, x3));
}

// Sum / max over the whole wave.
__device__ __forceinline__ float sum64(float x) {
  x = sum32(x);
  uint32_t a, b;
  pair32(__float_as_uint(x), a, b);
  return __uint_as_float(a) + __uint_as_float(b);
}
__device__ __forceinline__ float max64(float x) {
  x = fmaxf(x, dpp<kDppXor1>(x));
  x = fmaxf(x, dpp<kDppXor2>(x));
  x = fmaxf(x, dpp<kDppRor4>(x));
  x = fmaxf(x, dpp<kDppRor8>(x));
  uint32_t a, b;
  pair16(__float_as_uint(x), a, b);
  x = fmaxf(__uint_as_float(a), __uint_as_float(b));
  pair32(__float_as_uint(x), a, b);
  return fmaxf(__uint_as_float(a), __uint_as_float(b));
}

// x[l] op x[l ^ 32] in every lane with one v_permlane32_swap (no LDS round
// trip): swapping the wave's halves hands each lane the pair {x[l], x[l ^ 32]}.
__device__ __forceinline__ float sum_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Map a 1-D block id to a logical work id so that each of the 8 XCDs (which
// receive blocks round-robin) works on one contiguous range of logical ids and
// its private L2 sees a coherent working set.  The grid must be a multiple of 8
// blocks; ids >= n are padding and must exit.
__device__ __forceinline__ int64_t xcd_swizzle(int64_t bid, int64_t grid) {
  const int64_t per = grid >> 3;
  return (bid & 7) * per + (bid >> 3);
}

// Work order of the persistent query-chunk streams (S = streams per XCD; the
// item list is (b, h, c) in order).
// * Ranges (default): XCD x owns the x-th eighth of the items and its streams
//   sweep that range side by side (stream t takes items lo + t, lo + t + S, ...),
//   so each XCD works on a run of consecutive query chunks of one (batch, head)
//   slice and carries its L2 contents from one run to the next; the eight XCDs'
//   slices together are the last-level cache's working set.
// * Windows: the chip sweeps the items in windows of 8 S consecutive items;
//   within window r, XCD x takes the S items of part (x + r) mod 8.  The whole
//   chip then works on one slice at a time, for slices whose key/value chunks,
//   eight at once, would not fit the last-level cache; the rotation deals every
//   XCD the early (short-history) and late parts of the windows alike.
struct StreamOrder {
  int64_t S, st, lo, hi;  // streams per XCD; this stream within its XCD; the XCD's range
  int64_t nwork;
  int xcd;
  bool windows;
  __device__ __forceinline__ StreamOrder(int64_t S_, int64_t st_, int xcd_, int64_t nwork_, bool windows_)
      : S(S_), st(st_), lo(nwork_ * xcd_ / 8), hi(nwork_ * (xcd_ + 1) / 8), nwork(nwork_), xcd(xcd_),
        windows(windows_) {}
  __device__ __forceinline__ int64_t item(int64_t r) const {
    return windows ? (r * 8 + ((xcd + r) & 7)) * S + st : lo + st + r * S;
  }
  // number of items of this stream (items grow with r)
  __device__ __forceinline__ int64_t length() const {
    if (!windows) return lo + st < hi ? (hi - lo - st + S - 1) / S : 0;
    const int64_t full = nwork / (8 * S);
    return full + (item(full) < nwork ? 1 : 0);
  }
};

// The window order pays when the key/value chunks of eight (batch, head) slices
// (one per XCD under the range order) exceed the 256 MiB last-level cache.
inline bool use_window_order(int64_t nKV, size_t elem_bytes) {
  const int64_t slice_bytes = nKV * (int64_t)(2 * kS * kD) * (int64_t)elem_bytes;
  return 8 * slice_bytes > (int64_t(256) << 20);
}

// Position (b, h, c) of work item w = (b * H + h) * nQ + c, advanced a fixed
// number of chunks at a time so that persistent loops need no divisions.
struct Geo {
  int64_t b, c;
  int h;
  __device__ __forceinline__ Geo(int64_t w, int64_t nQ, int H) {
    c = w % nQ;
    const int64_t bh = w / nQ;
    h = (int)(bh % H);
    b = bh / H;
  }
  __device__ __forceinline__ void next(int64_t nQ, int H, int64_t step) {
    c += step;
    while (c >= nQ) {
      c -= nQ;
      if (++h == H) {
        h = 0;
        ++b;
      }
    }
  }
};

// ---------------------------------------------------- top-k selection ----

// ------------------------------------------------------- Gumbel noise ----
//
// Gumbel top-k retrieval adds g = -ln(-ln u) to every candidate's score before
// the selection (and only there).  u comes from the Philox4x32-10 counter-based
// generator (Salmon et al., SC 2011): key = the 64-bit seed, counter = (j / 4,
// t, b * Hr + hr, 0) for candidate chunk j of landmark row t, output word j mod
// 4, whose top 24 bits x give u = (x + 1/2) / 2^24 (exact in fp32).
__device__ __forceinline__ uint32_t philox_word(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                                uint32_t k1, int word) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint32_t lo0 = 0xD2511F53u * c0, hi0 = __umulhi(0xD2511F53u, c0);
    const uint32_t lo1 = 0xCD9E8D57u * c2, hi1 = __umulhi(0xCD9E8D57u, c2);
    c0 = hi1 ^ c1 ^ k0;
    c1 = lo1;
    c2 = hi0 ^ c3 ^ k1;
    c3 = lo0;
  }
  return word == 0 ? c0 : word == 1 ? c1 : word == 2 ? c2 : c3;
}

// g for candidate chunk j of landmark row t in (batch, retrieval head) slice bhr.
// The logarithms are v_log_f32 (base 2) scaled by ln 2.
__device__ __forceinline__ float gumbel_noise(uint64_t seed, uint32_t bhr, uint32_t t, uint32_t j) {
  const uint32_t x = philox_word(j >> 2, t, bhr, 0u, (uint32_t)seed, (uint32_t)(seed >> 32), (int)(j & 3));
  const float u = ((float)(x >> 8) + 0.5f) * 5.9604644775390625e-8f;  // 2^-24
  const float e = -kLn2 * __builtin_amdgcn_logf(u);                   // -ln u > 0
  return -kLn2 * __builtin_amdgcn_logf(e);
}

// The four values of candidates 4 j4 .. 4 j4 + 3 (one generator call).
__device__ __forceinline__ f32x4 gumbel_noise4(uint64_t seed, uint32_t bhr, uint32_t t, uint32_t j4) {
  uint32_t c0 = j4, c1 = t, c2 = bhr, c3 = 0u, k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint32_t lo0 = 0xD2511F53u * c0, hi0 = __umulhi(0xD2511F53u, c0);
    const uint32_t lo1 = 0xCD9E8D57u * c2, hi1 = __umulhi(0xCD9E8D57u, c2);
    c0 = hi1 ^ c1 ^ k0;
    c1 = lo1;
    c2 = hi0 ^ c3 ^ k1;
    c3 = lo0;
  }
  const uint32_t x[4] = {c0, c1, c2, c3};
  f32x4 g;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float u = ((float)(x[w] >> 8) + 0.5f) * 5.9604644775390625e-8f;
    g[w] = -kLn2 * __builtin_amdgcn_logf(-kLn2 * __builtin_amdgcn_logf(u));
  }
  return g;
}

// fp32 dot product of two D-element rows (D a multiple of 8).
template <typename T>
__device__ __forceinline__ float dot_rows(const T* __restrict__ a, const T* __restrict__ b, int D) {
  float acc = 0.f;
  for (int x = 0; x < D; x += 8) {
    const Frag<T> fa = load_frag(a + x), fb = load_frag(b + x);
#pragma unroll
    for (int m = 0; m < 8; ++m) acc = fmaf(frag_elem(fa, m), frag_elem(fb, m), acc);
  }
  return acc;
}

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

// Wave-wide best of one (score, chunk) per lane (every lane gets it).
__device__ __forceinline__ void take_better(float& s, int& j, float os, int oj) {
  if (better(os, oj, s, j)) {
    s = os;
    j = oj;
  }
}

// A candidate as one 64-bit key that orders like `better`: the score's bits made
// order-preserving (sign bit set for non-negative scores, all bits flipped for
// negative ones; -0 is taken as +0) above the complemented chunk index, so the
// larger key is the better candidate and the empty entry (-inf, kNoChunk) is
// below every real one.
__device__ __forceinline__ uint64_t pack_key(float s, int j) {
  uint32_t u = s == 0.f ? 0u : __float_as_uint(s);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)u << 32) | (uint64_t)(~(uint32_t)j);
}
__device__ __forceinline__ float key_score(uint64_t k) {
  const uint32_t u = (uint32_t)(k >> 32);
  return __uint_as_float((u & 0x80000000u) ? (u & 0x7fffffffu) : ~u);
}
__device__ __forceinline__ int key_chunk(uint64_t k) { return (int)~(uint32_t)k; }

// A lane's running best-KM list as packed candidate keys (pack_key), sorted
// largest first; 0 marks an empty entry (below every real key).  One insert is
// KM 64-bit compares against the old entries and a shift by selects.
template <int KM>
struct TopKeys {
  uint64_t k[KM];

  __device__ __forceinline__ void init() {
#pragma unroll
    for (int i = 0; i < KM; ++i) k[i] = 0;
  }
  __device__ __forceinline__ void insert(uint64_t x) {
    bool b[KM];
#pragma unroll
    for (int i = 0; i < KM; ++i) b[i] = x > k[i];
#pragma unroll
    for (int i = KM - 1; i > 0; --i) k[i] = b[i - 1] ? k[i - 1] : (b[i] ? x : k[i]);
    k[0] = b[0] ? x : k[0];
  }
};

template <int CTRL>
__device__ __forceinline__ uint64_t dpp64(uint64_t x) {
  return (uint64_t)dpp<CTRL>((uint32_t)x) | ((uint64_t)dpp<CTRL>((uint32_t)(x >> 32)) << 32);
}
__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }
// Wave-wide maximum key (every lane gets it).
__device__ __forceinline__ uint64_t wave_max_key(uint64_t k) {
  k = umax64(k, dpp64<kDppXor1>(k));
  k = umax64(k, dpp64<kDppXor2>(k));
  k = umax64(k, dpp64<kDppRor4>(k));
  k = umax64(k, dpp64<kDppRor8>(k));
  uint32_t l0, l1, h0, h1;
  pair16((uint32_t)k, l0, l1);
  pair16((uint32_t)(k >> 32), h0, h1);
  k = umax64((uint64_t)l0 | ((uint64_t)h0 << 32), (uint64_t)l1 | ((uint64_t)h1 << 32));
  pair32((uint32_t)k, l0, l1);
  pair32((uint32_t)(k >> 32), h0, h1);
  return umax64((uint64_t)l0 | ((uint64_t)h0 << 32), (uint64_t)l1 | ((uint64_t)h1 << 32));
}

// x of lane l ^ 4 (within each 32-lane half): ds_swizzle in bit-mask mode,
// lane l reads lane ((l & 31) ^ 4).
__device__ __forceinline__ uint32_t swz_xor4(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_ds_swizzle((int)x, 0x1F | (4 << 10));
}

// Bitonic sort of one key per lane across the wave, largest first: lane r
// receives the r-th largest key.  Stage (size kk, distance j) pairs lane l with
// l ^ j; inside a block whose bit kk is clear the lower lane keeps the larger
// key, inside the others the smaller, so the final stage leaves one descending
// run.  Distances 16 and 32 use the permlane swaps, which hand every lane both
// keys of its pair, so the kept key is their max or min.
__device__ __forceinline__ uint64_t wave_sort_desc(uint64_t k) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int kk = 2; kk <= 64; kk <<= 1) {
#pragma unroll
    for (int j = kk >> 1; j > 0; j >>= 1) {
      const bool keep_max = ((lane & j) == 0) == ((lane & kk) == 0);
      uint64_t a, b;
      if (j == 16 || j == 32) {
        uint32_t l0, l1, h0, h1;
        if (j == 16) {
          pair16((uint32_t)k, l0, l1);
          pair16((uint32_t)(k >> 32), h0, h1);
        } else {
          pair32((uint32_t)k, l0, l1);
          pair32((uint32_t)(k >> 32), h0, h1);
        }
        a = (uint64_t)l0 | ((uint64_t)h0 << 32);
        b = (uint64_t)l1 | ((uint64_t)h1 << 32);
      } else {
        a = k;
        if (j == 1) b = dpp64<kDppXor1>(k);
        else if (j == 2) b = dpp64<kDppXor2>(k);
        else if (j == 4) b = (uint64_t)swz_xor4((uint32_t)k) | ((uint64_t)swz_xor4((uint32_t)(k >> 32)) << 32);
        else b = dpp64<kDppRor8>(k);  // j == 8: rotating a 16-lane row by 8 pairs l with l ^ 8
      }
      k = ((a > b) == keep_max) ? a : b;  // the larger key where the lane keeps the max
    }
  }
  return k;
}

// Keys sorted largest first across the wave (lane r: r-th) in wave_merge's form:
// lane r < count holds the r-th best of the first k.
__device__ __forceinline__ void sorted_keys_top(uint64_t key, int k, float& my_s, int& my_j, int& count) {
  const int lane = threadIdx.x & 63;
  const bool real = key_chunk(key) != kNoChunk;
  count = __popcll(__ballot(real && lane < k));
  my_s = lane < count ? key_score(key) : -INFINITY;
  my_j = lane < count ? key_chunk(key) : kNoChunk;
}

// The wave's best k (k <= 64) when every lane holds at most one candidate
// (empty lanes pass -inf / kNoChunk), in wave_merge's form.
__device__ __forceinline__ void wave_top_one(float s, int j, int k, float& my_s, int& my_j, int& count) {
  sorted_keys_top(wave_sort_desc(pack_key(s, j)), k, my_s, my_j, count);
}

// The wave's best k (k <= 32) of two candidates per lane: both columns sorted,
// then the best 32 of each (column 1's moved to lanes 32-63) sorted together.
__device__ __forceinline__ void wave_top_two(uint64_t a, uint64_t b, int k, float& my_s, int& my_j, int& count) {
  const int lane = threadIdx.x & 63;
  a = wave_sort_desc(a);
  b = wave_sort_desc(b);
  // lane l >= 32 takes b of lane l - 32: the permlane swap hands every lane both
  // keys of its pair (l, l ^ 32); the one that is not its own is the partner's
  uint32_t l0, l1, h0, h1;
  pair32((uint32_t)b, l0, l1);
  pair32((uint32_t)(b >> 32), h0, h1);
  const uint64_t r0 = (uint64_t)l0 | ((uint64_t)h0 << 32), r1 = (uint64_t)l1 | ((uint64_t)h1 << 32);
  const uint64_t other = r0 != b ? r0 : r1;
  sorted_keys_top(wave_sort_desc(lane < 32 ? a : other), k, my_s, my_j, count);
}

// Merge the 64 lanes' lists into the wave's best k (k <= 64).  Lane r < *count
// receives the r-th best (score, chunk); *count <= k is the number of real
// candidates.  Lists are consumed.  Each round takes the wave's best list head
// as one 64-bit maximum.
template <int KM>
__device__ __forceinline__ void wave_merge(TopList<KM>& L, int k, float& my_s, int& my_j, int& count) {
  const int lane = threadIdx.x & 63;
  my_s = -INFINITY;
  my_j = kNoChunk;
  count = 0;
  for (int r = 0; r < k; ++r) {
    const uint64_t own = pack_key(L.s[0], L.j[0]);
    const uint64_t best = wave_max_key(own);
    const int bj = key_chunk(best);
    if (bj == kNoChunk) break;
    if (own == best) L.pop();
    if (lane == r) {
      my_s = key_score(best);
      my_j = bj;
    }
    ++count;
  }
}

// Merge of NW waves' results (lane r < cnt: the wave's r-th best, r < 32) by
// wave 0, which receives the workgroup's best (<= K <= 32) as wave_merge leaves
// it.  sS/sJ hold NW * 32 entries, sCnt NW.  Contains a workgroup barrier.
template <int KM, int NW>
__device__ __forceinline__ void merge_wave_results(int K, float* sS, int* sJ, int* sCnt, float& ms, int& mj,
                                                   int& cnt) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane < 32) {
    sS[wave * 32 + lane] = ms;
    sJ[wave * 32 + lane] = mj;
  }
  if (lane == 0) sCnt[wave] = cnt;
  __syncthreads();
  if (wave == 0) {
    if (NW * K <= 64) {
      // one candidate per lane: lane l takes entry l % K of wave l / K
      const int w = lane / K, r = lane - w * K;
      const bool has = w < NW && r < sCnt[w < NW ? w : 0];
      const int at = has ? w * 32 + r : 0;
      const float cs = sS[at];
      const int cj = sJ[at];
      wave_top_one(has ? cs : -INFINITY, has ? cj : kNoChunk, K, ms, mj, cnt);
    } else {
      TopList<KM> L;
      L.init();
#pragma unroll
      for (int w0 = 0; w0 < NW; w0 += 2) {
        const int w = w0 + (lane >> 5);  // lanes 0-31 take wave w0, lanes 32-63 wave w0 + 1
        if (w < NW && (lane & 31) < sCnt[w]) L.insert(sS[w * 32 + (lane & 31)], sJ[w * 32 + (lane & 31)]);
      }
      wave_merge(L, K, ms, mj, cnt);
    }
  }
}

// The decode scan's lists: scan workgroup g covers chunks [4 g pw, 4 (g + 1) pw)
// in groups of 8 consecutive chunks, its wave w taking groups w, w + 4, w + 8, ...
// (the four waves stream one contiguous range side by side) and leaving list
// 4 g + w.  The list that holds chunk c:
constexpr int kScanListWaves = 4;
__device__ __forceinline__ int64_t scan_list_of(int64_t c, int64_t pw) {
  const int64_t span = kScanListWaves * pw;
  return (c / span) * kScanListWaves + ((c % span) / 8) % kScanListWaves;
}

// Best k (<= 32) of one retrieval row from the decode scan's lists: list l (of
// `lists`) holds the best k of its chunks (scan_list_of), sorted best first and
// padded with chunk -1, at ls/lj[(row * lists + l) * K ..].  Every wave takes a
// contiguous share of the lists and the best k of their maxima; an entry of the
// row's top k can only sit in a list whose maximum is among the k best of its
// share (k better maxima would all beat it), so the wave merges the k-lists of
// those lists, and wave 0 merges the waves' results.  Result in wave 0 as
// wave_merge leaves it.  Scratch: sS/sJ/sCnt as merge_wave_results.
template <int KM, int NW>
__device__ void merge_lists(const float* __restrict__ ls, const int* __restrict__ lj, int64_t row, int64_t lists,
                            int64_t pw, int K, float* sS, int* sJ, int* sCnt, float& ms, int& mj, int& cnt) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float* rs = ls + row * lists * K;
  const int* rj = lj + row * lists * K;
  const int64_t share = (lists + NW - 1) / NW;
  const int64_t l_lo = wave * share, l_hi = l_lo + share < lists ? l_lo + share : lists;
  TopList<KM> L;
  L.init();
  // 1. the best k of the share's list maxima
  if (share <= 128 && K <= 32) {
    uint64_t c[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t l = l_lo + 64 * u + lane;
      const bool ok = l < l_hi;
      const int64_t lc = ok ? l : 0;
      const float v = rs[lc * K];
      const int j = rj[lc * K];
      c[u] = pack_key(ok && j >= 0 ? v : -INFINITY, ok && j >= 0 ? j : kNoChunk);
    }
    wave_top_two(c[0], c[1], K, ms, mj, cnt);
  } else {
    // four loads per lane in flight, running lists
    for (int64_t l0 = l_lo; l0 < l_hi; l0 += 256) {
      float v[4];
      int j[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int64_t l = l0 + 64 * u + lane;
        const int64_t lc = l < l_hi ? l : l_lo;
        v[u] = rs[lc * K];
        j[u] = l < l_hi ? rj[lc * K] : -1;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (j[u] >= 0) L.insert(v[u], j[u]);
    }
    wave_merge(L, K, ms, mj, cnt);
  }
  // 2. the k entries of each list they head (entry e: list e / K, rank e % K)
  const int ne = cnt * K;
  if (K * K <= 64) {
    float cs = -INFINITY;
    int cj = kNoChunk;
    const int src = lane / K;
    const int head = __shfl(mj, src);  // every lane takes part in the exchange
    if (lane < ne) {
      const int64_t l = scan_list_of(head, pw);
      const int64_t off = l * K + (lane - src * K);
      const int jj = rj[off];
      if (jj >= 0) {
        cs = rs[off];
        cj = jj;
      }
    }
    wave_top_one(cs, cj, K, ms, mj, cnt);
  } else {
    L.init();
    for (int e = lane; e < ne; e += 64) {
      const int src = e / K;
      const int64_t l = scan_list_of(__shfl(mj, src), pw);
      const int64_t off = l * K + (e - src * K);
      const int jj = rj[off];
      if (jj >= 0) L.insert(rs[off], jj);
    }
    wave_merge(L, K, ms, mj, cnt);
  }
  // 3. across the waves
  merge_wave_results<KM, NW>(K, sS, sJ, sCnt, ms, mj, cnt);
}

// Position of lane r's chunk among the first `count` lanes' chunks in
// ascending chunk order (chunks are distinct).
__device__ __forceinline__ int rank_by_chunk(int my_j, int count) {
  int rank = 0;
  for (int r = 0; r < count; ++r) {
    const int oj = __builtin_amdgcn_readlane(my_j, r);
    rank += (oj < my_j) ? 1 : 0;
  }
  return rank;
}

// Fusion weights (Eq. 2) of one retrieval row computed by one wave: lane s < K
// loads slot s; returns w (0 on pads) and the chunk (-1 on pads) in that lane,
// and whether the row has any valid slot.  Valid slots are 0 <= idx < nKV.
__device__ __forceinline__ bool wave_row_weight(const int32_t* __restrict__ idx, const float* __restrict__ sel,
                                                int64_t row_off, int K, int64_t nKV, float& w, int& j) {
  const int lane = threadIdx.x & 63;
  int jj = -1;
  float sv = -INFINITY;
  if (lane < K) {
    jj = idx[row_off + lane];
    sv = sel[row_off + lane];
  }
  const bool valid = lane < K && jj >= 0 && jj < nKV;
  float m = valid ? sv : -INFINITY;
  m = max64(m);
  const bool any = __ballot(valid) != 0;
  const float e = valid ? expf(sv - m) : 0.f;
  float sum = e;
  sum = sum64(sum);
  w = valid ? e / sum : 0.f;
  j = valid ? jj : -1;
  return any;
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
