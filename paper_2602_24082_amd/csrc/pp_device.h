// Device helpers for the gfx950 (CDNA4) kernels: bf16 vector types, loads that
// round fp32 inputs to bf16, the 32x32x16 bf16 MFMA and its register layout.
//
// v_mfma_f32_32x32x16_bf16 (wave64) computes D[32x32] += A[32x16] * B[16x32]:
//   A operand: lane l holds A[m = l%32][k = 8*(l/32) + e], e = 0..7
//   B operand: lane l holds B[k = 8*(l/32) + e][n = l%32], e = 0..7
//   D/C:       lane l holds D[m = 8*(r/4) + 4*(l/32) + r%4][n = l%32], r = 0..15
// Both operands therefore read 8 consecutive elements along the contraction
// axis, and the result's column n is owned by lanes l and l+32.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_huge_valf();

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// 2^x on the hardware transcendental unit (v_exp_f32): exp2(-inf) = 0, results
// below the normal range flush toward 0, which is harmless for softmax weights.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}

// 8 consecutive elements as bf16 (fp32 input is rounded to nearest even).
template <typename T>
__device__ __forceinline__ bf16x8 load8_bf16(const T* p);

template <>
__device__ __forceinline__ bf16x8 load8_bf16<__bf16>(const __bf16* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}

template <>
__device__ __forceinline__ bf16x8 load8_bf16<float>(const float* p) {
  const f32x4 a = *reinterpret_cast<const f32x4*>(p);
  const f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
  f32x8 x = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return __builtin_convertvector(x, bf16x8);
}

// Stores 4 consecutive outputs in the tensor's element type.
template <typename T>
__device__ __forceinline__ void store4(T* p, f32x4 v);

template <>
__device__ __forceinline__ void store4<__bf16>(__bf16* p, f32x4 v) {
  *reinterpret_cast<bf16x4*>(p) = __builtin_convertvector(v, bf16x4);
}

template <>
__device__ __forceinline__ void store4<float>(float* p, f32x4 v) {
  *reinterpret_cast<f32x4*>(p) = v;
}

__device__ __forceinline__ bf16x8 to_bf16x8(float a0, float a1, float a2, float a3, float a4, float a5,
                                             float a6, float a7) {
  f32x8 x = {a0, a1, a2, a3, a4, a5, a6, a7};
  return __builtin_convertvector(x, bf16x8);
}

// The 16 accumulator registers r = 8s..8s+7 (s = 0, 1) of a 32x32 result, as a
// bf16 B operand of a K=16 MFMA.  Lane half h = l/32 then holds rows
// 16s + 8*(e/4) + 4h + e%4 for e = 0..7, i.e. the contraction index
// kk = 8h + e stands for row 16s + perm16(kk) with
//   perm16(kk) = 8*((kk%8)/4) + 4*(kk/8) + kk%4.
// An A operand read from LDS must use the same row order (see lds_tr8).
__device__ __forceinline__ bf16x8 acc_half_to_bf16(const f32x16& acc, int s) {
  return to_bf16x8(acc[8 * s + 0], acc[8 * s + 1], acc[8 * s + 2], acc[8 * s + 3], acc[8 * s + 4],
                   acc[8 * s + 5], acc[8 * s + 6], acc[8 * s + 7]);
}

// ---------------------------------------------------------------------------
// LDS tiles: [rows][D] bf16, rows packed back to back (D*2 bytes), with the
// 16-byte chunks of row r XOR-swizzled by swz<D>(r).  The swizzle is a bijection
// on every aligned group of 16 rows, so 16-byte reads of one logical chunk down
// 16 consecutive rows hit 16 different bank groups; and the four rows x four
// chunks that a half-wave touches in a transposed read also land in distinct
// bank groups.  Tiles are filled by global_load_lds_dwordx4 (lane l of a wave
// writes 16 bytes at the wave's LDS base + 16*l), so each lane fetches the
// global chunk that belongs at its swizzled position.
// ---------------------------------------------------------------------------

typedef __attribute__((address_space(3))) void lds_void;

// One global_load_lds_dwordx4: lane l's 16 bytes at `src` land at LDS byte
// address `lds_dst` (wave-uniform, passed through M0) + 16*l.  Every kernel
// waits for these explicitly (wait_vmem / wait_tile) before the barrier that
// publishes a stage, and reads a stage only after that barrier.
//
// The instruction is issued as inline assembly rather than through the
// compiler builtin.  The compiler cannot tell which LDS bytes an LDS DMA
// writes, so after the builtin it waits for every outstanding DMA before the
// next LDS read it cannot prove disjoint (in practice the first transposed
// read of each tile) -- which includes the prefetch of the NEXT tile and so
// serialises the prefetch with half of the compute it should overlap.  The
// kernels' own waits are exact; the "memory" clobber keeps the compiler from
// moving LDS accesses across the statement.  The LDS base goes in as an M0
// operand, so the compiler sets M0 itself and knows what it holds.
__device__ __forceinline__ void lds_dma16(const void* src, const void* lds_dst) {
  const unsigned base = __builtin_amdgcn_readfirstlane((unsigned)(uintptr_t)(lds_void*)lds_dst);
  asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(base) : "memory");
}

// One 4-byte element per lane into LDS (lane l -> lds + 4*l): the per-query
// scalars of a 64-query tile.  Issued like lds_dma16.
__device__ __forceinline__ void dma_dword(void* lds, const void* src) {
  const unsigned base = __builtin_amdgcn_readfirstlane((unsigned)(uintptr_t)(lds_void*)lds);
  asm volatile("global_load_lds_dword %0, off" ::"v"(src), "{m0}"(base) : "memory");
}
typedef short i16x4 __attribute__((ext_vector_type(4)));

template <int D>
__device__ __forceinline__ int swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}

// Wave-cooperative DMA of NR tile rows [row0, row0 + NR) into LDS.  Tile row r
// comes from `src + min(r, rows_valid - 1) * stride` (elements), so rows past
// the valid range repeat the last valid row (finite data that the mask then
// ignores).  NR * D * 2 must be a multiple of 1 KB.  The per-lane part of the
// addresses is a 32-bit byte offset computed once (`init`); `issue` adds it to
// the wave-uniform tile base, which the loads take from scalar registers.
template <int D, int NR>
struct TileDma {
  static constexpr int RPI = 1024 / (D * 2);  // rows per wave instruction
  static constexpr int CPR = D / 8;           // 16-byte chunks per row
  static constexpr int N = NR / RPI;          // instructions per call
  static_assert(NR % RPI == 0, "tile rows must fill whole wave loads");
  uint32_t off[N];  // byte offset of this lane's chunk in instruction i, full tile
  uint32_t stride_b;  // bytes between tile rows
  int row0;
  int lane;

  // tile row and 16-byte chunk (of the swizzled row) that this lane fetches in instruction i
  __device__ __forceinline__ int row_of(int i) const { return row0 + i * RPI + lane / CPR; }
  __device__ __forceinline__ uint32_t chunk_b(int i) const { return (uint32_t)((lane % CPR) ^ swz<D>(row_of(i))) << 4; }

  __device__ __forceinline__ void init(int row0_, int64_t stride_, int lane_) {
    row0 = row0_;
    stride_b = (uint32_t)(stride_ * 2);
    lane = lane_;
#pragma unroll
    for (int i = 0; i < N; ++i) off[i] = (uint32_t)row_of(i) * stride_b + chunk_b(i);
  }

  __device__ __forceinline__ void issue(__bf16* lds_tile, const __bf16* src, int rows_valid) const {
    const char* base = reinterpret_cast<const char*>(src);
    if (rows_valid >= row0 + N * RPI) {
#pragma unroll
      for (int i = 0; i < N; ++i) lds_dma16(base + off[i], lds_tile + (row0 + i * RPI) * D);
    } else {
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const uint32_t rs = (uint32_t)min(row_of(i), rows_valid - 1);
        lds_dma16(base + (rs * stride_b + chunk_b(i)), lds_tile + (row0 + i * RPI) * D);
      }
    }
  }
};

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt in bits 3:0 and 15:14, expcnt 6:4 and lgkmcnt 11:8 left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// 16-byte read of logical chunk `lc` (elements 8*lc .. 8*lc+7) of tile row r.
template <int D>
__device__ __forceinline__ bf16x8 lds_row8(const __bf16* tile, int r, int lc) {
  return *reinterpret_cast<const bf16x8*>(tile + r * D + ((lc ^ swz<D>(r)) << 3));
}

// A operand of a 32x32x16 MFMA whose A[m][k] = tile[row(k)][col0 + m], i.e. the
// tile read transposed: m runs along the row (d) axis, k along tile rows.  The
// contraction index kk = 8h + e (h = lane/32) stands for tile row
// row16 + perm16(kk): rows row16 + 4h + 0..3 for e < 4 and row16 + 8 + 4h + 0..3
// for e >= 4, which is the order in which a 32x32 accumulator's registers hold
// their rows (see acc_half_to_bf16).  Two ds_read_b64_tr_b16: in each group of
// 16 lanes, lane 4r+q addresses 4 consecutive columns of row r and the hardware
// returns to lane i the column i of the 4 rows.
template <int D>
__device__ __forceinline__ bf16x8 lds_tr8(const __bf16* tile, int row16, int col0, int lane) {
  const int g = lane >> 4, a = lane & 15;
  const int r = a >> 2, q = a & 3;
  const int h = g >> 1;
  const int col = col0 + 16 * (g & 1) + 4 * q;
  const int lc = col >> 3, sub = col & 7;
  const int r0 = row16 + 4 * h + r;
  const int r1 = r0 + 8;
  const __bf16* p0 = tile + r0 * D + ((lc ^ swz<D>(r0)) << 3) + sub;
  const __bf16* p1 = tile + r1 * D + ((lc ^ swz<D>(r1)) << 3) + sub;
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p0);
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p1);
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, v);
}

// A 32 x 32 bf16 tile of dS as the backward stores it: 32 key rows of 64
// bytes, no swizzle.  The key-major pass (lane = key) writes a lane pair's two
// accumulator halves side by side, so column c of a row holds query
// ds_query_of_column(c) of the block: bits (c4 c3 c2 c1 c0) -> (c3 c2 c4 c1 c0),
// the order in which a 32x32 accumulator's registers hold their rows.
__device__ __forceinline__ int ds_query_of_column(int c) {
  return 16 * ((c >> 3) & 1) + 8 * ((c >> 2) & 1) + 4 * (c >> 4) + (c & 3);
}

// B operand of a 32x32x16 MFMA from such a tile read transposed: lane l gets
// column l % 32 of rows row16 + perm16(kk) (the row order of lds_tr8).  Each
// ds_read_b64_tr_b16 covers eight whole 64-byte rows: no bank conflicts.
__device__ __forceinline__ bf16x8 lds_tr8_tile32(const __bf16* tile, int row16, int lane) {
  const int g = lane >> 4, a = lane & 15;
  const int r0 = row16 + 4 * (g >> 1) + (a >> 2);
  const int col = 16 * (g & 1) + 4 * (a & 3);
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(tile + r0 * 32 + col));
  const i16x4 hi =
      __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(tile + (r0 + 8) * 32 + col));
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  i16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  return __builtin_bit_cast(bf16x8, v);
}

// The lane's index in its wave, formed where it is used (v_mbcnt from no
// input register; volatile, so the compiler neither hoists it out of a loop
// nor keeps it live across one -- under full register pressure it spilled
// such a value and reloaded it with a wait that also covered the tile DMAs).
__device__ __forceinline__ int lane_id_here() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// Workgroup barrier that orders LDS accesses only (s_waitcnt lgkmcnt(0);
// s_barrier): global stores issued before it stay in flight, where
// __syncthreads would wait for them.  LDS filled by DMA is published by an
// explicit wait_vmem ahead of it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Waits until pipelined tile t has landed, given that tiles t+1 ..
// min(t+NS-2, n-1) (each PER_TILE DMA instructions of this wave, issued after
// tile t) may still be in flight.  Vector-memory loads complete in order.
template <int NS, int PER_TILE>
__device__ __forceinline__ void wait_tile(int t, int n) {
  if constexpr (NS == 2) {
    wait_vmem<0>();
  } else if constexpr (NS == 3) {
    if (t + 1 < n) wait_vmem<PER_TILE>();
    else wait_vmem<0>();
  } else {
    static_assert(NS == 4, "pipeline depth 2, 3 or 4");
    if (t + 2 < n) wait_vmem<2 * PER_TILE>();
    else if (t + 1 < n) wait_vmem<PER_TILE>();
    else wait_vmem<0>();
  }
}

// max / sum of x and the value held by lane l ^ 32 (the other half of the
// wave), through v_permlane32_swap: a VALU exchange of the two 32-lane halves
// of two registers, with no LDS round trip.  Swapping x with itself leaves
// r[0] = x of lane l & 31 and r[1] = x of lane (l & 31) + 32 in every lane.
__device__ __forceinline__ float half_swap_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float a = __uint_as_float(r[0]), b = __uint_as_float(r[1]);
  return a > b ? a : b;
}
__device__ __forceinline__ float half_swap_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float wave_max(float x) {
  for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

// Instruction classes of __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedValu = 0x002;
constexpr int kSchedMfma = 0x008;
constexpr int kSchedDsRead = 0x100;
constexpr int kSchedTrans = 0x400;

// Visibility bitmasks of a lane's row of a block: bit o is set when the
// block's o-th element in that row is visible.  A lane forms its mask once per
// block from a few ranges; each element is then kept or set to -inf by one
// signed bit extract and one bit insert, instead of compares and selects.
__device__ __forceinline__ uint64_t bits_below64(int n) {  // bits [0, n), n of any sign
  return n <= 0 ? 0ull : n >= 64 ? ~0ull : ((1ull << n) - 1ull);
}
__device__ __forceinline__ uint32_t bits_below32(int n) {
  return n <= 0 ? 0u : n >= 32 ? ~0u : ((1u << n) - 1u);
}
// x where bit `bit` of `word` is set, else -inf
__device__ __forceinline__ float keep_or_neginf(float x, uint32_t word, int bit) {
  const int m = __builtin_amdgcn_sbfe((int)word, bit, 1);  // 0 or -1
  return __int_as_float((__float_as_int(x) & m) | (~m & (int)0xff800000u));
}

// Wave-wide any of a lane predicate, as a value the compiler knows is uniform
// (so a branch on it does not make a loop divergent).
__device__ __forceinline__ bool wave_any(bool x) { return __builtin_amdgcn_readfirstlane(__any(x)) != 0; }

// A read-only plan record at a wave-uniform address, fetched with scalar loads
// (through the constant address space) so that it lands in scalar registers
// and is waited for on the scalar counter.  A vector load would be followed by
// a wait on the vector-memory counter, which also waits for every LDS DMA
// issued before it, including prefetches meant to stay in flight.
// Each 32-bit field is loaded on its own: an aggregate copy is lowered to
// loads the backend keeps on the vector path.
__device__ __forceinline__ int32_t scalar_load(const int32_t* p) {
  return *(const __attribute__((address_space(4))) int32_t*)p;
}

template <typename Item>
__device__ __forceinline__ Item load_uniform(const Item* p) {
  static_assert(sizeof(Item) % 4 == 0, "plan records are made of 32-bit fields");
  Item out;
  const int32_t* src = reinterpret_cast<const int32_t*>(p);
  int32_t* dst = reinterpret_cast<int32_t*>(&out);
#pragma unroll
  for (int i = 0; i < (int)(sizeof(Item) / 4); ++i) dst[i] = scalar_load(src + i);
  return out;
}

// cos and sin of the rotary angle pos * inv_freq.  The angle is formed in fp64
// and reduced there to r in [-pi/4, pi/4] plus a quadrant k (angle = k pi/2 + r),
// so the result does not depend on the size of the position (an fp32 product of
// a position near 8192 would already be off by ~5e-4 rad).  sin r and cos r are
// their Taylor series through r^9 and r^10, evaluated in fp32 (truncation below
// 2e-9 on the interval); the quadrant then permutes and negates them.
__device__ __forceinline__ void rope_cos_sin(int pos, double inv_freq, float& c, float& s) {
  const double a = (double)pos * inv_freq;
  const double k = rint(a * 0.6366197723675814);  // 2 / pi
  const float r = (float)fma(-k, 1.5707963267948966, a);
  const float r2 = r * r;
  const float sr = r * (1.f + r2 * (-1.f / 6 + r2 * (1.f / 120 + r2 * (-1.f / 5040 + r2 * (1.f / 362880)))));
  const float cr =
      1.f + r2 * (-0.5f + r2 * (1.f / 24 + r2 * (-1.f / 720 + r2 * (1.f / 40320 + r2 * (-1.f / 3628800)))));
  const int q = (int)((int64_t)k & 3);
  const float ss = (q & 1) ? cr : sr;
  const float cc = (q & 1) ? sr : cr;
  s = (q & 2) ? -ss : ss;
  c = (q == 1 || q == 2) ? -cc : cc;
}

// Maps a linear workgroup index to (item, head).  Workgroups are dispatched to
// the 8 XCDs round-robin (index % 8); when the head count is a multiple of 8 the
// heads of one item are arranged so that each XCD receives a contiguous run of
// heads, which for grouped-query attention is one kv-head's query group, so its
// K/V tiles are shared through that XCD's L2.
__device__ __forceinline__ void item_and_head(int block, int heads, int& item, int& head) {
  item = block / heads;
  const int r = block - item * heads;
  if ((heads & 7) == 0) {
    const int per = heads >> 3;
    head = (r & 7) * per + (r >> 3);
  } else {
    head = r;
  }
}

}  // namespace pp
