// Grouped expert GEMMs of the chunked MoE layer on gfx950 matrix cores.
//
// Every GEMM of the expert SwiGLU FFN and its backward (the "expert" of the
// paper's Eq. (4) and its derivative in Eq. (5); Table 2 rows 11-13 name the
// tensors) is written as
//     C[m, n] = sum_kk A(m, kk) * B(n, kk)
// over one expert at a time and multiplied by 32x32 MFMA instructions
// (v_mfma_f32_32x32x16_bf16, or v_mfma_f32_32x32x2f32 on the fp32 path).
//
// Operand movement.  Operand tiles go from HBM into LDS directly with
// buffer_load ... lds (16 bytes per lane, no staging registers), or, as a
// launch option, through registers (buffer_load into VGPRs during the
// previous K tile's multiply, then ds_write_b128).  Buffer resources bound
// each tensor, so rows past
// the end of a tensor, ragged tails and the K tail of a weight-gradient tile
// read as zero in hardware.
// Two LDS layouts serve the two ways an operand can sit in HBM:
//   K-contiguous  ([row][k], 128-byte K rows): activation rows, weights used
//                 as W^T.  Rows may be gathered through the chunk's
//                 row -> token table, so dispatch never materialises a
//                 permuted copy of X or dY.  Read with ds_read_b128.
//   K-strided     ([k][row], one HBM row per k): weights used as W, and both
//                 operands of the weight gradients, whose reduction axis is
//                 the expert's rows.  Read with two ds_read_b64_tr_b16, which
//                 transpose 4 K rows x 16 columns across each 16-lane group
//                 into the K-packed MFMA operand (fp32: a plain 4-byte read).
// Both layouts XOR-swizzle 16-byte units so that the lanes of one LDS read
// instruction hit distinct banks.
//
// Tiling.  A workgroup of WM x WN waves owns a BM x BN output tile; each
// wave owns (BM/WM) x (BN/WN) as 32 x 32 MFMA blocks whose accumulators stay
// in registers for the whole K loop.  The default is 256 x 256 on 8 waves
// (2 x 4, 128 x 64 per wave, two waves per SIMD, one workgroup per CU);
// 128 x 128 tiles serve problems whose 256 x 256 grid would leave CUs idle
// and the quarter-tile tail of a launch.  K tiles (128 bytes of K per
// operand row) are double-buffered in 128 KB of LDS: the copy of tile k+1
// runs while the waves multiply tile k, with one barrier per K step.
//
// Tile order.  Workgroups are dealt round-robin to the 8 XCDs; the
// row-grouped GEMMs map ids to tiles in blocks of 32 per XCD (8 m-tiles x 4
// n-tiles) so that the tiles one XCD holds at once share operand K-slices in
// its L2, and launches
// of equal-cost direct-copy tiles run persistent (one workgroup per CU, the
// next tile's first copies in flight during the epilogue).
//
// Scheduling on skewed expert loads: the row-grouped GEMMs (forward FC1/FC2,
// dgrads) enumerate m-tiles expert after expert from the chunk's offsets, so
// a cold expert costs only its own ceil(rows/BM) tiles; the weight-gradient
// GEMMs (K = the expert's rows) visit experts in descending row count, the
// longest tiles first.
#include "common.h"
#include "kernels.h"

namespace memfine {
namespace {


constexpr uint32_t kOOB = 0x80000000u;    // byte offset past every buffer's range
#ifndef MEMFINE_SCHED_HINTS
#define MEMFINE_SCHED_HINTS 1
#endif
constexpr bool kSchedHints = MEMFINE_SCHED_HINTS;
// Wave priority while a tile's MFMAs issue (s_setprio), for the
// register-staged copy loop: there each wave also issues the next K tile's
// loads and LDS writes, and the SIMD's arbiter then favours the wave that
// feeds the matrix core (3-6 % faster; the direct-copy loops measured 1-2 %
// slower with it, so they keep the default priority).
#ifndef MEMFINE_MMA_PRIO
#define MEMFINE_MMA_PRIO 2
#endif
constexpr int kMmaPrio = MEMFINE_MMA_PRIO;
// The direct-copy loops instead raise it from the K step's wait through the
// barrier and the issue of the next K tile's copies, so that the copies go
// out before the other wave's MFMAs take the issue slots (-0.3-0.4 % step
// time; priority during their MFMAs measured 1-2 % slower).
#ifndef MEMFINE_DIRECT_PRIO
#define MEMFINE_DIRECT_PRIO 1
#endif
constexpr int kDirectPrio = MEMFINE_DIRECT_PRIO;
// Carry each K tile's last MFMA step over the next K step's barrier (see
// mma_tile_carry) in the direct-copy loops.
#ifndef MEMFINE_CARRY_STEP
#define MEMFINE_CARRY_STEP 1
#endif
constexpr bool kCarryStep = MEMFINE_CARRY_STEP;
// Weight gradients adding into dW: 1 = the epilogue loads the old values and
// adds them to the tile's sum; 0 = the accumulators start from them, loaded
// before the tile's first MFMA (that wait also waits for the previous tile's
// stores, which the next tile's first K steps otherwise hide).
#ifndef MEMFINE_DW_ADD_IN_EPILOGUE
#define MEMFINE_DW_ADD_IN_EPILOGUE 1
#endif
constexpr bool kDwAddInEpilogue = MEMFINE_DW_ADD_IN_EPILOGUE;
// s_waitcnt lgkmcnt(0): this wave's LDS reads have returned
__device__ __forceinline__ void wait_lgkm0() {
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
}

typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4;

// Tile shape: BM x BN output per workgroup of WM x WN waves, S LDS stages of
// KB bytes of K per operand row.  DIRECT_ bit 0 (operand A) and bit 1
// (operand B): the operand's tiles go from HBM straight into LDS
// (buffer_load ... lds); else through registers (buffer_load into VGPRs
// during the multiply of the previous tile, then ds_write_b128).
template <int BM_, int BN_, int WM_, int WN_, int S_, int KB_ = 128, int DIRECT_ = 3> struct Cfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, S = S_, KB = KB_;
  static constexpr bool DA = (DIRECT_ & 1) != 0, DB = (DIRECT_ & 2) != 0;
  static constexpr bool DIRECT = DA && DB;  // both direct: the deeper-stage loop
  static constexpr int NW = WM * WN, kThreads = 64 * NW;
  static constexpr int WTM = BM / WM, WTN = BN / WN;  // wave tile
  static constexpr int MB = WTM / 32, NB = WTN / 32;  // 32x32 MFMA blocks per wave
  static constexpr int kStage = (BM + BN) * KB;
  static constexpr int kLds = S * kStage;
  static constexpr int kWgPerCu = (160 * 1024) / kLds;
  static constexpr int kMinWaves = (kWgPerCu * NW + 3) / 4 < 3 ? (kWgPerCu * NW + 3) / 4 : 3;
  // Wave w's block of the tile.  Waves w and w + 4 of a workgroup share a
  // SIMD (checked on the GPU with HW_ID).  On the 2 x 4 grid the two waves
  // of a SIMD take different wave rows and column halves (w < 4: (0, w);
  // w >= 4: (1, (w + 2) % 4)), so that a tile whose lower half of rows or
  // right half of columns lies past the data still keeps every SIMD's
  // matrix core busy with the other wave's blocks (see `active`).
  __device__ __forceinline__ static void wave_role(int w, int& wm, int& wn) {
    if constexpr (WM == 2 && WN == 4) {
      wm = w >> 2;
      wn = (w + 2 * (w >> 2)) & 3;
    } else {
      wm = w / WN;
      wn = w % WN;
    }
  }
};
using Small = Cfg<128, 128, 2, 2, 2>;

// Epilogue staging.  Straight from the accumulators, a 16-byte store
// instruction would touch 32 rows (one per lane pair) in 8- or 16-byte
// pieces.  Bounced through a wave-private LDS slab of 32 rows x 128 bytes
// (16-byte units XOR-swizzled by row), each instruction writes 8 rows x 128
// contiguous bytes instead.  The slabs sit after the stages (wave w at
// kLds + w * kSlabBytes), where the LDS has room without costing a
// workgroup per CU.
constexpr int kSlabBytes = 32 * 128;
template <class C> constexpr int kSlabArea =
    (C::kLds + C::NW * kSlabBytes) * C::kWgPerCu <= 160 * 1024 ? C::NW * kSlabBytes : 0;
// Slab per wave taken from the stages by epilogues that run with no copies
// in flight.
constexpr int kStageSlabBytes = 8 * 1024;
// kArray: bytes of the LDS array the tile runs in (0: a launch of C's own,
// sized C::kLds + kSlabArea<C>)
template <class C, int kArray = 0> __device__ __forceinline__ char* slab_of(char* smem, int wave) {
  constexpr bool fits = kArray > 0 ? C::kLds + C::NW * kSlabBytes <= kArray : kSlabArea<C> > 0;
  if constexpr (fits) return smem + C::kLds + wave * kSlabBytes;
  else return nullptr;
}

// Tile order.  Workgroup ids are dealt round-robin to the 8 XCDs (XCD x
// runs ids x, x + 8, ...), and the workgroups an XCD holds at once share its
// L2.  Operand K-slices that several resident tiles read are then fetched
// from memory once; tiles spread over all XCDs instead read the same slices
// into every XCD's L2, and the copies wait on the Infinity Fabric.  So for
// raster > 0 workgroup ids map to logical tiles in blocks of 32 consecutive
// tiles per XCD (one workgroup per CU, 32 CUs per XCD): block b goes to XCD
// b % 8.  Alternating blocks between XCDs keeps their loads even where tile
// costs drift along the order (weight gradients walk the experts in
// descending row count).  Ids past the last whole round of 256 keep their
// index.  The map is a bijection of [0, n).
__device__ __forceinline__ int xcd_block_remap(int id, int n) {
  if (id >= (n & ~255)) return id;
  const int x = id & 7, slot = id >> 3;
  return ((slot >> 5) << 8) | (x << 5) | (slot & 31);
}
// Groups of `group` m-tiles, m fastest inside a group; all n-tiles of a group
// before the next group.  A bijection of [0, mtn * ntn) onto the grid.
__device__ __forceinline__ void grouped_coords(int logical, int mtn, int ntn, int group, int& mt,
                                               int& nt) {
  const int per_group = group * ntn;
  const int g = logical / per_group;
  const int first_m = g * group;
  const int gsz = min(mtn - first_m, group);
  const int r = logical - g * per_group;
  mt = first_m + r % gsz;
  nt = r / gsz;
}
// Logical tile of workgroup `id` among the n workgroups that share the grid.
__device__ __forceinline__ int logical_of(int raster, int id, int n) {
  return raster <= 0 ? id : xcd_block_remap(id, n);
}
// Coordinates of logical tile L on an mtn x ntn grid: raster 0 and 4
// row-major (n-tiles fastest), 1..3 groups of 4 << (raster - 1) m-tiles.
__device__ __forceinline__ void logical_coords(int raster, int L, int mtn, int ntn, int& mt,
                                               int& nt) {
  if (raster >= 1 && raster <= 3) {
    grouped_coords(L, mtn, ntn, 4 << (raster - 1), mt, nt);
  } else {
    mt = L / ntn;
    nt = L % ntn;
  }
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const int32_t n = (int32_t)(bytes < (int64_t)kOOB ? bytes : (int64_t)kOOB - 1);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}
// a range the caller knows to be below 2^31 bytes (no clamp)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc32(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int32_t)bytes,
                                           0x00020000);
}

__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t r, char* lds, uint32_t voff,
                                           uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)lds, 16, voff, soff, 0, 0);
}
__device__ __forceinline__ u32x4_t load_reg16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
}
// 16-byte store; an offset past the resource's range is dropped by the
// hardware, so the instruction issues whatever the lane's element is
__device__ __forceinline__ void store_f32x4(__amdgpu_buffer_rsrc_t r, uint32_t voff, const float (&v)[4]) {
  f32x4_t x;
#pragma clang loop unroll(full)
  for (int c = 0; c < 4; ++c) x[c] = v[c];
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, x), r, voff, 0, 0);
}

// 4 floats as 4 bf16 (8 bytes)
__device__ __forceinline__ u32x2_t pack4(const float (&f)[4]) {
  u32x2_t x;
  x[0] = pack_bf16x2(f[0], f[1]);
  x[1] = pack_bf16x2(f[2], f[3]);
  return x;
}

template <typename T> struct Mma;
template <> struct Mma<bf16_t> {
  static constexpr int kKStep = 16;
  typedef bf16x8_t Frag;
  __device__ __forceinline__ static void mma(const Frag& a, const Frag& b, f32x16_t& c) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mma<float> {
  static constexpr int kKStep = 2;
  typedef float Frag;
  __device__ __forceinline__ static void mma(const Frag& a, const Frag& b, f32x16_t& c) {
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

// --------------------------------------------------------- K-contiguous
// LDS tile: ROWS rows x KB bytes (KB = 64 or 128, i.e. U = 4 or 8 units of
// 16 bytes); unit c of row r sits at unit c ^ sw(r), which puts the 8 rows
// that one LDS cycle serves on distinct banks.  The direct copy writes 1 KB
// (1024 / KB rows) per wave instruction: lane l lands at physical unit
// l % U of row l / U, so it fetches the logical unit (l % U) ^ sw(row).
template <int KB> __device__ __forceinline__ int kc_sw(int row) {
  if constexpr (KB == 128) return (row ^ (row >> 3)) & 7;
  else return (row >> 1) & 3;
}
template <int KB> __device__ __forceinline__ int kc_off(int row, int c) {
  return row * KB + ((c ^ kc_sw<KB>(row)) << 4);
}
template <int KB, int ROWS>
__device__ __forceinline__ bf16x8_t kc_read_bf16(const char* lds, int row0, int kk, int lane) {
  const int row = row0 + (lane & 31);
  return *(const bf16x8_t*)(lds + kc_off<KB>(row, kk * 2 + (lane >> 5)));
}
template <int KB, int ROWS>
__device__ __forceinline__ float kc_read_f32(const char* lds, int row0, int kk, int lane) {
  const int row = row0 + (lane & 31);
  const int kel = kk * 2 + (lane >> 5);
  return *(const float*)(lds + kc_off<KB>(row, kel >> 2) + ((kel & 3) << 2));
}

template <typename T, int ROWS, int NW, int KB, bool DIRECT> struct KcOp {
  static constexpr int kReadsPerFrag = 1;
  static constexpr int U = KB / 16;          // 16-byte units per row
  static constexpr int RPI = 1024 / KB;      // rows per copy instruction
  static constexpr int I = ROWS / (RPI * NW);  // copy instructions per wave per K tile
  static_assert(I * RPI * NW == ROWS, "tile rows must split evenly over the waves");
  __amdgpu_buffer_rsrc_t rs;
  uint32_t voff[I];
  u32x4_t stage[DIRECT ? 1 : I];  // register-staged copy of one K tile
  __device__ __forceinline__ static int row_of(int i, int wave, int lane) {
    return RPI * (i * NW + wave) + lane / U;
  }
  // row_byte(row) -> byte offset of the row's first K element, or kOOB
  template <class F> __device__ __forceinline__ void init(F row_byte, int wave, int lane) {
#pragma clang loop unroll(full)
    for (int i = 0; i < I; ++i) {
      const int row = row_of(i, wave, lane);
      const uint32_t rb = row_byte(row);
      // direct copies land at lane * 16, so the swizzle picks the global unit;
      // staged copies fetch the row's units in order and swizzle on the write
      const int unit = DIRECT ? ((lane % U) ^ kc_sw<KB>(row)) : lane % U;
      voff[i] = rb == kOOB ? kOOB : rb + (uint32_t)(unit << 4);
    }
  }
  __device__ __forceinline__ void issue(char* lds, int kt, int wave) {
#pragma clang loop unroll(full)
    for (int i = 0; i < I; ++i) {
      if constexpr (DIRECT) load_lds16(rs, lds + (i * NW + wave) * 1024, voff[i], kt * KB);
      else stage[i] = load_reg16(rs, voff[i], kt * KB);
    }
  }
  // register-staged copy: unit lane % U of the row goes to its swizzled place
  __device__ __forceinline__ void commit(char* lds, int wave, int lane) const {
    if constexpr (!DIRECT) {
#pragma clang loop unroll(full)
      for (int i = 0; i < I; ++i)
        *(u32x4_t*)(lds + kc_off<KB>(row_of(i, wave, lane), lane % U)) = stage[i];
    }
  }
  __device__ __forceinline__ static typename Mma<T>::Frag read(const char* lds, int row0, int kk,
                                                               int lane) {
    if constexpr (sizeof(T) == 2) return kc_read_bf16<KB, ROWS>(lds, row0, kk, lane);
    else return kc_read_f32<KB, ROWS>(lds, row0, kk, lane);
  }
};

// ------------------------------------------------------------ K-strided
// LDS tile: BK rows (one per k) of ROWS elements (pitch P = ROWS * size);
// 16-byte unit u of k-row k sits at unit u ^ ks_sw(k).  The swizzle spreads
// the 4 consecutive k-rows that one transposing read touches over distinct
// banks.  A copy instruction writes 1 KB = 1024 / P whole k-rows.
__device__ __forceinline__ int ks_sw(int k) {
  // k & 3 = 0, 1, 2, 3  ->  units 0, 10, 4, 14 (branch-free)
  return ((k & 1) * 10) ^ ((k & 2) * 2);
}

template <typename T, int ROWS, int NW, int KB, bool DIRECT> struct KsOp {
  static constexpr int kReadsPerFrag = sizeof(T) == 2 ? 2 : 1;
  static constexpr int BKE = KB / (int)sizeof(T);  // k-rows per K tile
  static constexpr int P = ROWS * (int)sizeof(T);
  static constexpr int KPI = 1024 / P;          // k-rows per copy instruction
  static constexpr int I = BKE / (KPI * NW);      // copy instructions per wave per K tile
  static_assert(I * KPI * NW == BKE, "K tile must split evenly over the waves");
  static constexpr int V = 16 / (int)sizeof(T); // elements per 16-byte unit
  __amdgpu_buffer_rsrc_t rs;
  uint32_t voff[I];
  u32x4_t stage[DIRECT ? 1 : I];  // register-staged copy of one K tile
  // lane's k-row (within the K tile) and logical element column of instruction i
  __device__ __forceinline__ static int k_of(int i, int wave, int lane) {
    return (i * NW + wave) * KPI + (lane * 16) / P;
  }
  // logical element column fetched by the lane (direct copies swizzle here,
  // staged copies on the LDS write)
  __device__ __forceinline__ static int col_of(int i, int wave, int lane) {
    const int k = k_of(i, wave, lane);
    const int p = ((lane * 16) % P) >> 4;
    return (DIRECT ? (p ^ ks_sw(k)) : p) * V;
  }
  __device__ __forceinline__ void issue(char* lds, uint32_t soff, int wave) {
#pragma clang loop unroll(full)
    for (int i = 0; i < I; ++i) {
      if constexpr (DIRECT) load_lds16(rs, lds + (i * NW + wave) * 1024, voff[i], soff);
      else stage[i] = load_reg16(rs, voff[i], soff);
    }
  }
  __device__ __forceinline__ void commit(char* lds, int wave, int lane) const {
    if constexpr (!DIRECT) {
      const int p = ((lane * 16) % P) >> 4;
#pragma clang loop unroll(full)
      for (int i = 0; i < I; ++i) {
        const int k = k_of(i, wave, lane);
        *(u32x4_t*)(lds + k * P + ((p ^ ks_sw(k)) << 4)) = stage[i];
      }
    }
  }
  __device__ __forceinline__ static int phys(int k, int col) {  // byte of element col in k-row
    const int b = col * (int)sizeof(T);
    return k * P + ((((b >> 4) ^ ks_sw(k))) << 4) + (b & 15);
  }
  __device__ __forceinline__ static typename Mma<T>::Frag read(const char* lds, int col0, int kk,
                                                               int lane);
};
// k-row k, element column col: byte offset inside a K-strided tile of pitch P
template <int P, int ES>
__device__ __forceinline__ int ks_phys(int k, int col) {
  const int b = col * ES;
  return k * P + ((((b >> 4) ^ ks_sw(k))) << 4) + (b & 15);
}
// `lds` is restrict: inlined, the transposing reads then carry alias-scope
// information, without which the compiler makes every LDS read wait for all
// direct-to-LDS copies in flight (those of the next K tile included, which
// write the other stage); the K loop's own waits and barriers order the
// copies and the reads.
template <int ROWS>
__device__ __forceinline__ bf16x8_t ks_read_bf16(const char* __restrict__ lds, int col0, int kk,
                                                 int lane) {
  // MFMA lane l wants column col0 + l%32 and K values 8*(l/32) .. +7.  In the
  // 16-lane group G = l/16, source lane j supplies 4 columns starting at
  // col0 + 16*(G%2) + 4*(j%4) of k-row 16 kk + 8*(G/2) + 4h + j/4; after the
  // transpose, lane j of the group holds that column's 4 consecutive k.
  const int j = lane & 15, G = lane >> 4;
  const int col = col0 + (G & 1) * 16 + 4 * (j & 3);
  const int k0 = kk * 16 + (G >> 1) * 8 + (j >> 2);
  const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_s16x4*)(lds + ks_phys<ROWS * 2, 2>(k0, col)));
  const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_s16x4*)(lds + ks_phys<ROWS * 2, 2>(k0 + 4, col)));
  return __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}
template <int ROWS>
__device__ __forceinline__ float ks_read_f32(const char* lds, int col0, int kk, int lane) {
  return *(const float*)(lds + ks_phys<ROWS * 4, 4>(kk * 2 + (lane >> 5), col0 + (lane & 31)));
}
template <typename T, int ROWS, int NW, int KB, bool DIRECT>
__device__ __forceinline__ typename Mma<T>::Frag KsOp<T, ROWS, NW, KB, DIRECT>::read(const char* lds, int col0,
                                                                       int kk, int lane) {
  if constexpr (sizeof(T) == 2) return ks_read_bf16<ROWS>(lds, col0, kk, lane);
  else return ks_read_f32<ROWS>(lds, col0, kk, lane);
}
// --------------------------------------------------------------- compute
template <class C> struct Accum {
  f32x16_t v[C::MB][C::NB];
};
template <class C> __device__ __forceinline__ void zero_acc(Accum<C>& acc) {
#pragma clang loop unroll(full)
  for (int i = 0; i < C::MB; ++i)
#pragma clang loop unroll(full)
    for (int j = 0; j < C::NB; ++j)
#pragma clang loop unroll(full)
      for (int q = 0; q < 16; ++q) acc.v[i][j][q] = 0.f;
}

// One K tile: the operand fragments of K step kk+1 are read from LDS while
// the MFMAs of step kk run (two fragment register sets); scheduling
// barriers interleave the LDS reads with the MFMAs so that neither waits
// on the other.
template <typename T, class C, class OA, class OB>
__device__ __forceinline__ void mma_tile(const char* As, const char* Bs, Accum<C>& acc, int wm,
                                         int wn, int lane) {
  constexpr int KS = C::KB / (int)sizeof(T) / Mma<T>::kKStep;
  constexpr int kReads = OA::kReadsPerFrag * C::MB + OB::kReadsPerFrag * C::NB;
  constexpr int kMfma = C::MB * C::NB;
  typename Mma<T>::Frag a[2][C::MB], b[2][C::NB];
  constexpr int kPrio = C::DIRECT ? 0 : kMmaPrio;
  if constexpr (kPrio > 0) __builtin_amdgcn_s_setprio(kPrio);
#pragma clang loop unroll(full)
  for (int i = 0; i < C::MB; ++i) a[0][i] = OA::read(As, wm * C::WTM + i * 32, 0, lane);
#pragma clang loop unroll(full)
  for (int j = 0; j < C::NB; ++j) b[0][j] = OB::read(Bs, wn * C::WTN + j * 32, 0, lane);
#pragma clang loop unroll(full)
  for (int kk = 0; kk < KS; ++kk) {
    const int cu = kk & 1, nx = cu ^ 1;
    if (kk + 1 < KS) {
      // B's fragments first: every MFMA of a row i uses all of them, A's
      // fragment i only its own row
#pragma clang loop unroll(full)
      for (int j = 0; j < C::NB; ++j) b[nx][j] = OB::read(Bs, wn * C::WTN + j * 32, kk + 1, lane);
#pragma clang loop unroll(full)
      for (int i = 0; i < C::MB; ++i) a[nx][i] = OA::read(As, wm * C::WTM + i * 32, kk + 1, lane);
    }
#pragma clang loop unroll(full)
    for (int i = 0; i < C::MB; ++i)
#pragma clang loop unroll(full)
      for (int j = 0; j < C::NB; ++j) Mma<T>::mma(b[cu][j], a[cu][i], acc.v[i][j]);
  }
  if constexpr (kSchedHints) {
    // DS reads of step 0, then per step: MFMAs of step kk interleaved with the
    // reads of step kk+1, then the MFMAs of the last step.
    __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
#pragma clang loop unroll(full)
    for (int kk = 0; kk + 1 < KS; ++kk) {
#pragma clang loop unroll(full)
      for (int x = 0; x < kMfma; ++x) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if (kReads <= kMfma) {
          if (x < kReads) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        } else {
          // more reads than MFMAs (the weight gradients' two transposed
          // operands): all of them go out during this step's MFMAs, the
          // surplus with the first ones, so that none waits at the step's end
          __builtin_amdgcn_sched_group_barrier(0x100, kReads / kMfma, 0);
          if (x < kReads % kMfma) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
      }
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kMfma, 0);
  }
  if constexpr (kPrio > 0) __builtin_amdgcn_s_setprio(0);
}

// One K tile whose last MFMA step is carried over: its fragments stay in
// registers (set 1) and its MFMAs are issued by the next call (kCarry)
// after the next K step's barrier, where they cover that tile's first
// fragment reads, or by mma_flush after the K loop.
template <typename T, class C> struct FragSets {
  typename Mma<T>::Frag a[2][C::MB], b[2][C::NB];
};
template <typename T, class C, class OA, class OB, bool kCarry>
__device__ __forceinline__ void mma_tile_carry(const char* As, const char* Bs, Accum<C>& acc, int wm,
                                               int wn, int lane, FragSets<T, C>& f) {
  constexpr int KS = C::KB / (int)sizeof(T) / Mma<T>::kKStep;
  static_assert(KS % 2 == 0, "the carried step uses fragment set 1");
  constexpr int kReads = OA::kReadsPerFrag * C::MB + OB::kReadsPerFrag * C::NB;
  constexpr int kMfma = C::MB * C::NB;
  constexpr int kPrio = C::DIRECT ? 0 : kMmaPrio;  // as in mma_tile
  if constexpr (kPrio > 0) __builtin_amdgcn_s_setprio(kPrio);
#pragma clang loop unroll(full)
  for (int i = 0; i < C::MB; ++i) f.a[0][i] = OA::read(As, wm * C::WTM + i * 32, 0, lane);
#pragma clang loop unroll(full)
  for (int j = 0; j < C::NB; ++j) f.b[0][j] = OB::read(Bs, wn * C::WTN + j * 32, 0, lane);
  if constexpr (kCarry) {
#pragma clang loop unroll(full)
    for (int i = 0; i < C::MB; ++i)
#pragma clang loop unroll(full)
      for (int j = 0; j < C::NB; ++j) Mma<T>::mma(f.b[1][j], f.a[1][i], acc.v[i][j]);
  }
#pragma clang loop unroll(full)
  for (int kk = 0; kk + 1 < KS; ++kk) {
    const int cu = kk & 1, nx = cu ^ 1;
    // B's fragments first, as in mma_tile
#pragma clang loop unroll(full)
    for (int j = 0; j < C::NB; ++j) f.b[nx][j] = OB::read(Bs, wn * C::WTN + j * 32, kk + 1, lane);
#pragma clang loop unroll(full)
    for (int i = 0; i < C::MB; ++i) f.a[nx][i] = OA::read(As, wm * C::WTM + i * 32, kk + 1, lane);
#pragma clang loop unroll(full)
    for (int i = 0; i < C::MB; ++i)
#pragma clang loop unroll(full)
      for (int j = 0; j < C::NB; ++j) Mma<T>::mma(f.b[cu][j], f.a[cu][i], acc.v[i][j]);
  }
  if constexpr (kSchedHints) {
    // the carried MFMAs interleaved with step 0's reads, then per step the
    // MFMAs of step kk interleaved with the reads of step kk + 1
#pragma clang loop unroll(full)
    for (int kk = 0; kk < KS; ++kk) {
      if (kk == 0 && !kCarry) {
        __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
        continue;
      }
#pragma clang loop unroll(full)
      for (int x = 0; x < kMfma; ++x) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if (kReads <= kMfma) {
          if (x < kReads) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        } else {
          // more reads than MFMAs (the weight gradients' two transposed
          // operands): all of them go out during this step's MFMAs, the
          // surplus with the first ones, so that none waits at the step's end
          __builtin_amdgcn_sched_group_barrier(0x100, kReads / kMfma, 0);
          if (x < kReads % kMfma) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
      }
    }
  }
  if constexpr (kPrio > 0) __builtin_amdgcn_s_setprio(0);
}
template <typename T, class C>
__device__ __forceinline__ void mma_flush(Accum<C>& acc, const FragSets<T, C>& f) {
#pragma clang loop unroll(full)
  for (int i = 0; i < C::MB; ++i)
#pragma clang loop unroll(full)
    for (int j = 0; j < C::NB; ++j) Mma<T>::mma(f.b[1][j], f.a[1][i], acc.v[i][j]);
}

// Accumulator layout.  The MFMA is given the B fragment as its first operand,
// so block (mb, nb) holds the transposed product: element q of a lane sits at
// tile row acc_row(wm, mb, lane) and tile column acc_col(wn, nb, q / 4, lane)
// + q % 4.  Each lane thus owns one output row and four runs of four
// consecutive columns per block, which the epilogues move with 8- or 16-byte
// accesses.
template <class C> __device__ __forceinline__ int acc_row(int wm, int mb, int lane) {
  return wm * C::WTM + mb * 32 + (lane & 31);
}
template <class C> __device__ __forceinline__ int acc_col(int wn, int nb, int gq, int lane) {
  return wn * C::WTN + nb * 32 + gq * 8 + (lane >> 5) * 4;
}
// the four values of run gq of block acc
__device__ __forceinline__ void acc_run(const f32x16_t& acc, int gq, float (&f)[4]) {
#pragma clang loop unroll(full)
  for (int c = 0; c < 4; ++c) f[c] = acc[gq * 4 + c];
}

struct Tile {
  int e;      // expert
  int m0;     // first output row (row-grouped: chunk row; wgrad: weight row)
  int mrows;  // valid output rows in this tile
  int n0;     // first output column (FC1: first f)
  int K;      // reduction length
  int r0;     // wgrad: first chunk row of the expert
  int acc;    // wgrad: the accumulators start from the stored dW (add into it)
};

// m-tile bound for the row-grouped grid: sum_e ceil(c_e / BM) <= this.
inline int row_tiles_bound(int n, int E, int BM) {
  return (int)(((int64_t)n + (int64_t)E * (BM - 1)) / BM);
}

// A chunk's m-tiles of BM rows, expert after expert.  With at most 64
// experts one wave holds the whole table: lane e loads expert e's row range
// and a shuffle scan gives the inclusive prefix of the m-tile counts, so
// counting and locating tiles costs one load latency instead of a serial walk
// over the experts.  All lanes of the wave must call these together.
template <int BM> struct RowTiles {
  int o0 = 0, o1 = 0, n = 0, inc = 0, total = 0;
  __device__ __forceinline__ void load(const int32_t* __restrict__ offsets, int E) {
    const int lane = threadIdx.x & 63;
    if (lane < E) {
      o0 = offsets[lane];
      o1 = offsets[lane + 1];
    }
    n = (o1 - o0 + BM - 1) / BM;
    inc = n;
#pragma clang loop unroll(full)
    for (int d = 1; d < 64; d <<= 1) {
      const int v = __shfl_up(inc, d, 64);
      if (lane >= d) inc += v;
    }
    total = __builtin_amdgcn_readlane(inc, 63);
  }
  // expert and rows of m-tile mt; false past the last tile.  The results are
  // read into scalar registers (readlane): the buffer resources built from
  // them must be wave-uniform, or every copy becomes a waterfall loop.
  __device__ __forceinline__ bool locate(int mt, Tile& t) const {
    const unsigned long long m = __ballot(inc > mt);
    if (m == 0) return false;
    const int l = __builtin_ctzll(m);  // first expert whose tiles reach past mt
    const int before = __builtin_amdgcn_readlane(inc - n, l);
    t.e = l;
    t.m0 = __builtin_amdgcn_readlane(o0, l) + (mt - before) * BM;
    t.mrows = min(BM, __builtin_amdgcn_readlane(o1, l) - t.m0);
    return true;
  }
};

// m-tiles of a row-grouped grid: sum_e ceil(c_e / BM).
template <int BM> __device__ __forceinline__ int row_tiles(const int32_t* __restrict__ offsets, int E) {
  if (E <= 64) {
    RowTiles<BM> rt;
    rt.load(offsets, E);
    return rt.total;
  }
  int n = 0;
  for (int e = 0; e < E; ++e) n += (offsets[e + 1] - offsets[e] + BM - 1) / BM;
  return n;
}

// Expert and rows of m-tile `mt` of a row-grouped problem.
template <int BM>
__device__ __forceinline__ bool locate_rows(const int32_t* __restrict__ offsets, int E, int mt,
                                            Tile& t) {
  if (E <= 64) {
    RowTiles<BM> rt;
    rt.load(offsets, E);
    return rt.locate(mt, t);
  }
  int acc = 0;
  for (int e = 0; e < E; ++e) {
    const int r0 = offsets[e], r1 = offsets[e + 1];
    const int tiles = (r1 - r0 + BM - 1) / BM;
    if (mt < acc + tiles) {
      t.e = e;
      t.m0 = r0 + (mt - acc) * BM;
      t.mrows = min(BM, r1 - t.m0);
      return true;
    }
    acc += tiles;
  }
  return false;
}

// Row-grouped problems: output tiles of BM rows x BNU columns (P::ncols(g)
// columns in all), reduction length P::reduction(g).  Logical tile L of the
// chunk's grid of row_tiles x ntn tiles; false past the grid.
// m-tile and n-tile of logical tile L on the chunk's grid of BM-row m-tiles x
// ntn n-tiles, with the tile's expert and rows; false past the grid.
template <int BM>
__device__ __forceinline__ bool locate_grid(const GemmArgs& g, int L, int ntn, Tile& t, int& nt) {
  int mt;
  if (g.E <= 64) {
    RowTiles<BM> rt;
    rt.load(g.offsets, g.E);
    if (L >= rt.total * ntn) return false;
    logical_coords(g.raster, L, rt.total, ntn, mt, nt);
    return rt.locate(mt, t);
  }
  const int mtn = row_tiles<BM>(g.offsets, g.E);
  if (L >= mtn * ntn) return false;
  logical_coords(g.raster, L, mtn, ntn, mt, nt);
  return locate_rows<BM>(g.offsets, g.E, mt, t);
}
template <class P, int BM, int BNU>
__device__ __forceinline__ bool locate_row_logical(const GemmArgs& g, Tile& t, int L) {
  int nt;
  if (!locate_grid<BM>(g, L, (P::ncols(g) + BNU - 1) / BNU, t, nt)) return false;
  t.n0 = nt * BNU;
  t.K = P::reduction(g);
  return true;
}
// Workgroup id of the n that share the grid.
template <class P, int BM, int BNU>
__device__ __forceinline__ bool locate_row_tile(const GemmArgs& g, Tile& t, int id, int n) {
  return locate_row_logical<P, BM, BNU>(g, t, logical_of(g.raster, id, n));
}
// Quarter `sub` (2 x 2) of logical tile b of the grid with twice the tile
// size: the split tail of a launch.
template <class P, int BM, int BNU>
__device__ __forceinline__ bool locate_row_subtile(const GemmArgs& g, Tile& t, int b, int sub) {
  int nt;
  if (!locate_grid<2 * BM>(g, b, (P::ncols(g) + 2 * BNU - 1) / (2 * BNU), t, nt)) return false;
  const int sm = sub >> 1, sn = sub & 1;
  t.m0 += sm * BM;
  t.mrows = min(t.mrows - sm * BM, BM);
  t.n0 = (2 * nt + sn) * BNU;
  t.K = P::reduction(g);
  return t.mrows > 0 && t.n0 < P::ncols(g);
}
// Does wave (wm, wn) own any output of a row-grouped tile?  Its rows start
// at wm * WTM and its BNU / WN output columns at n0 + wn * BNU / WN.
template <class P, class C, int BNU>
__device__ __forceinline__ bool row_wave_active(const GemmArgs& g, const Tile& t, int wm, int wn) {
  return wm * C::WTM < t.mrows && t.n0 + wn * (BNU / C::WN) < P::ncols(g);
}

template <typename T> __device__ __forceinline__ const char* cptr(const void* base, int64_t el) {
  return (const char*)base + el * (int64_t)sizeof(T);
}

// Plain epilogue of a row-grouped problem: out[m0 + r, n0 + c] = acc, for
// an output of `ld` columns (ld % 64 == 0).
template <typename T, class C>
__device__ __forceinline__ void store_rows(const Accum<C>& acc, T* out, int ld, const Tile& t, int wm,
                                           int wn, int lane, char* slab = nullptr) {
  if constexpr (sizeof(T) == 2 && (C::WTN * 2) % 128 == 0) {
    if (slab != nullptr) {
      // bf16 rows of the wave's block in 128-byte column groups (64 columns,
      // two 32-column MFMA blocks); per (row block mb, group): the lanes write
      // their runs of row lane % 32 into the slab, then read back 16 bytes
      // each, 8 lanes to a row, and store 8 rows per instruction.  Elements
      // outside the tile get an offset past the resource (ld % 8 == 0: a
      // 16-byte unit is all in or all out).
      constexpr int CG = C::WTN * 2 / 128;
      const int m0 = __builtin_amdgcn_readfirstlane(t.m0);
      const int mrows = __builtin_amdgcn_readfirstlane(t.mrows);
      const int n0 = __builtin_amdgcn_readfirstlane(t.n0);
      const uint32_t rowb = (uint32_t)ld * 2;
      const __amdgpu_buffer_rsrc_t rs = make_rsrc(out + (int64_t)m0 * ld, (int64_t)mrows * rowb);
      const int rr = lane & 31, half = lane >> 5;
#pragma clang loop unroll(full)
      for (int mb = 0; mb < C::MB; ++mb)
#pragma clang loop unroll(full)
        for (int cg = 0; cg < CG; ++cg) {
#pragma clang loop unroll(full)
          for (int b = 0; b < 2; ++b)
#pragma clang loop unroll(full)
            for (int gq = 0; gq < 4; ++gq) {
              const int byte = b * 64 + gq * 16 + half * 8;  // run's byte in the 128-byte row
              float v[4];
              acc_run(acc.v[mb][cg * 2 + b], gq, v);
              u32x2_t x;
              x[0] = pack_bf16x2(v[0], v[1]);
              x[1] = pack_bf16x2(v[2], v[3]);
              *(u32x2_t*)(slab + rr * 128 + ((((byte >> 4) ^ (rr & 7))) << 4) + (byte & 15)) = x;
            }
          asm volatile("" ::: "memory");  // the writes above before the reads below
          const int unit = lane & 7;
#pragma clang loop unroll(full)
          for (int q = 0; q < 4; ++q) {
            const int r = (lane >> 3) + 8 * q;
            const u32x4_t x = *(const u32x4_t*)(slab + r * 128 + ((unit ^ (r & 7)) << 4));
            const int row = wm * C::WTM + mb * 32 + r;
            const int col = n0 + wn * C::WTN + cg * 64 + unit * 8;
            __builtin_amdgcn_raw_buffer_store_b128(
                x, rs, (row < mrows && col < ld) ? (uint32_t)row * rowb + (uint32_t)col * 2 : kOOB, 0,
                0);
          }
          asm volatile("" ::: "memory");  // the reads above before the next writes
        }
      return;
    }
  }
#pragma clang loop unroll(full)
  for (int mb = 0; mb < C::MB; ++mb) {
    const int r = acc_row<C>(wm, mb, lane);
    if (r >= t.mrows) continue;
    T* o = out + (int64_t)(t.m0 + r) * ld;
#pragma clang loop unroll(full)
    for (int nb = 0; nb < C::NB; ++nb)
#pragma clang loop unroll(full)
      for (int gq = 0; gq < 4; ++gq) {
        const int n = t.n0 + acc_col<C>(wn, nb, gq, lane);
        if (n >= ld) continue;
        float v[4];
        acc_run(acc.v[mb][nb], gq, v);
        Vec4<T>::store(o + n, v);
      }
  }
}

// ================================================================ problems
// Each problem provides locate (tile of this workgroup), init (buffer
// resources and per-lane copy offsets), issue (start the direct copies of one
// K tile into LDS), and epilogue (consume the accumulators).

// FC1 + SwiGLU, forward and the backward's recomputation of it.
//   A(m, kk) = X[tok(m0 + m), kk]            K = h  (gathered rows)
//   B(nr, kk) = W1[e, wrow(nr), kk]          each wave's WTN tile columns are
//   WTN/2 gate rows f followed by the WTN/2 up rows F + f of the same f, so
//   every lane holds both halves of its SwiGLU pairs (blocks nb, nb + NB/2).
// Forward epilogue: a = silu(u_g) u_u.  Backward epilogue (kBwd; dA = dY W2
// of the row is already in `ag`): with g the slot's gate and da = g dA,
//   du_g = da u_u silu'(u_g),  du_u = da silu(u_g)   -> u  [n, 2F]
//   g a                                              -> ag [n, F] (over dA)
//   dgp[m, f / 32] = sum over 32 columns f of dA a    (gate-gradient partials)
// Each dA element is read and then overwritten by the one lane that owns it.
template <typename T, class C, bool kBwd> struct ProbFC1 {
  typedef ProbFC1 ProbSelf;
  static constexpr bool kEqualTiles = true;  // every tile reduces over the same K
  static constexpr int kRaster = 2;  // preferred tile order (XCD blocks of 8 x 4 tiles)
  static constexpr bool kEpilogueLoads = kBwd;  // the epilogue reads global memory
  static constexpr int kHalf = C::WTN / 2;
  // the recomputation's epilogue can stage its stores through LDS (bf16, 32
  // output columns per wave)
  static constexpr bool kStaged = kBwd && sizeof(T) == 2 && kHalf == 32;
  typedef KcOp<T, C::BM, C::NW, C::KB, C::DA> OA;
  typedef KcOp<T, C::BN, C::NW, C::KB, C::DB> OB;
  OA A;
  OB B;
  static int grid(const GemmArgs& g) {
    return row_tiles_bound(g.n, g.E, C::BM) * ((ncols(g) + BNU - 1) / BNU);
  }
  static constexpr int BNU = C::BN / 2;  // output columns per tile
  __host__ __device__ static int ncols(const GemmArgs& g) { return g.F; }
  __device__ __forceinline__ bool locate(const GemmArgs& g, Tile& t, int id, int n) const {
    return locate_row_tile<ProbSelf, C::BM, BNU>(g, t, id, n);
  }
  __device__ __forceinline__ bool locate_sub(const GemmArgs& g, Tile& t, int b, int sub) const {
    return locate_row_subtile<ProbSelf, C::BM, BNU>(g, t, b, sub);
  }
  __device__ __forceinline__ static int total_tiles(const GemmArgs& g) {
    return row_tiles<C::BM>(g.offsets, g.E) * ((ncols(g) + BNU - 1) / BNU);
  }
  __device__ __forceinline__ bool active(const GemmArgs& g, const Tile& t, int wm, int wn) const {
    return row_wave_active<ProbSelf, C, BNU>(g, t, wm, wn);
  }
  __host__ __device__ static int reduction(const GemmArgs& g) { return g.h; }
  __device__ __forceinline__ void init(const GemmArgs& g, const Tile& t, int wave, int lane) {
    A.rs = make_rsrc(g.X, g.T_h_bytes);
    const int32_t* tok = g.tok_of_row + t.m0;
    const uint32_t rowb = (uint32_t)g.h * sizeof(T);
    A.init([&](int r) { return r < t.mrows ? (uint32_t)tok[r] * rowb : kOOB; }, wave, lane);
    B.rs = make_rsrc(cptr<T>(g.W1, (int64_t)t.e * 2 * g.F * g.h), (int64_t)2 * g.F * g.h * sizeof(T));
    B.init([&](int r) {
      const int w = r / C::WTN, q = r % C::WTN;
      const int f = t.n0 + w * kHalf + (q % kHalf);
      const int wrow = q >= kHalf ? g.F + f : f;
      return f < g.F ? (uint32_t)wrow * rowb : kOOB;
    }, wave, lane);
  }
  __device__ __forceinline__ void init_acc(const GemmArgs&, const Tile&, Accum<C>& acc, int, int,
                                          int) const {
    zero_acc(acc);
  }
  __device__ __forceinline__ void commit(char* As, char* Bs, int wave, int lane) const {
    A.commit(As, wave, lane);
    B.commit(Bs, wave, lane);
  }
  __device__ __forceinline__ void issue(const GemmArgs&, const Tile&, int kt, char* As, char* Bs,
                                        int wave, int) {
    A.issue(As, kt, wave);
    B.issue(Bs, kt, wave);
  }
  __device__ __forceinline__ void epilogue(const GemmArgs& g, const Tile& t, const Accum<C>& acc,
                                           int wm, int wn, int lane, char* slab) const {
    if constexpr (kBwd) {
      epilogue_bwd(g, t, acc, wm, wn, lane, slab);
    } else {
#pragma clang loop unroll(full)
      for (int mb = 0; mb < C::MB; ++mb) {
        const int r = acc_row<C>(wm, mb, lane);
        if (r >= t.mrows) continue;
        T* a = (T*)g.a + (t.m0 + r) * (int64_t)g.F;
#pragma clang loop unroll(full)
        for (int nb = 0; nb < C::NB / 2; ++nb)
#pragma clang loop unroll(full)
          for (int gq = 0; gq < 4; ++gq) {
            // F % 64 == 0: a run of 4 columns is entirely inside or outside
            const int f = t.n0 + wn * kHalf + nb * 32 + gq * 8 + (lane >> 5) * 4;
            if (f >= g.F) continue;
            float gate[4], up[4], act[4];
            acc_run(acc.v[mb][nb], gq, gate);
            acc_run(acc.v[mb][nb + C::NB / 2], gq, up);
#pragma clang loop unroll(full)
            for (int c = 0; c < 4; ++c) act[c] = gate[c] * sigmoidf_(gate[c]) * up[c];
            Vec4<T>::store(a + f, act);
          }
      }
    }
  }
  // Steps walk the row blocks mb; the dA values of block mb + 1 are loaded
  // while block mb is computed and stored (two buffers).  Rows past the tile
  // and column blocks past F load from clamped in-range addresses and are not
  // used.  With `slab` (bf16, 32 columns per wave: 3 x 2 KB per wave) the
  // three outputs of a row block go through it: the lanes write their runs
  // of row lane % 32 (64-byte rows, 16-byte units XOR-swizzled by row), then
  // read back 16 bytes each, 4 lanes to a row, and store 16 rows x 64 bytes
  // per instruction.
  __device__ __forceinline__ void epilogue_bwd(const GemmArgs& g, const Tile& t, const Accum<C>& acc,
                                               int wm, int wn, int lane, char* slab) const {
    typedef typename Vec4<T>::Raw Raw;
    constexpr int NH = C::NB / 2;  // gate (and up) blocks per wave
    Raw dar[2][NH][4];
    float gtb[2];
    auto fetch = [&](int mb, int b) {
      const int r = acc_row<C>(wm, mb, lane);
      const int64_t row = t.m0 + (r < t.mrows ? r : 0);
      gtb[b] = g.gate_of_row[row];
      const T* d = (const T*)g.ag + row * g.F;
#pragma clang loop unroll(full)
      for (int nb = 0; nb < NH; ++nb)
#pragma clang loop unroll(full)
        for (int gq = 0; gq < 4; ++gq) {
          const int f = t.n0 + wn * kHalf + nb * 32 + gq * 8 + (lane >> 5) * 4;
          dar[b][nb][gq] = Vec4<T>::load_raw(d + (f < g.F ? f : 0));
        }
    };
    fetch(0, 0);
#pragma clang loop unroll(full)
    for (int mb = 0; mb < C::MB; ++mb) {
      const int b = mb & 1;
      if (mb + 1 < C::MB) fetch(mb + 1, b ^ 1);
      const int r = acc_row<C>(wm, mb, lane);
      const bool in = r < t.mrows;
      const int64_t row = t.m0 + (in ? r : 0);
      const float gt = gtb[b];
      T* u = (T*)g.u + row * 2 * g.F;
      T* ag = (T*)g.ag + row * g.F;
#pragma clang loop unroll(full)
      for (int nb = 0; nb < NH; ++nb) {
        // F % 64 == 0 and the block starts at a multiple of 32: all or nothing
        const int fb = t.n0 + wn * kHalf + nb * 32;
        if (fb >= g.F) continue;
        float part = 0.f;
        const bool staged = kStaged && slab != nullptr;
#pragma clang loop unroll(full)
        for (int gq = 0; gq < 4; ++gq) {
          float dA[4], gate[4], up[4], dug[4], duu[4], ga[4];
          Vec4<T>::unpack(dar[b][nb][gq], dA);
          acc_run(acc.v[mb][nb], gq, gate);
          acc_run(acc.v[mb][nb + NH], gq, up);
#pragma clang loop unroll(full)
          for (int c = 0; c < 4; ++c) {
            const float x = gate[c], s = sigmoidf_(x), silu = x * s, act = silu * up[c];
            part = fmaf(dA[c], act, part);
            const float da = gt * dA[c];
            dug[c] = da * up[c] * s * (1.f + x * (1.f - s));
            duu[c] = da * silu;
            ga[c] = gt * act;
          }
          if (staged) {
            const int rr = lane & 31;
            const int off = rr * 64 + ((gq ^ (rr & 3)) << 4) + (lane >> 5) * 8;
            *(u32x2_t*)(slab + off) = pack4(dug);
            *(u32x2_t*)(slab + 2048 + off) = pack4(duu);
            *(u32x2_t*)(slab + 4096 + off) = pack4(ga);
          } else if (in) {
            const int f = fb + gq * 8 + (lane >> 5) * 4;
            Vec4<T>::store(u + f, dug);
            Vec4<T>::store(u + g.F + f, duu);
            Vec4<T>::store(ag + f, ga);
          }
        }
        if (staged) {
          asm volatile("" ::: "memory");  // the writes above before the reads below
          const int unit = lane & 3;
#pragma clang loop unroll(full)
          for (int o = 0; o < 3; ++o)
#pragma clang loop unroll(full)
            for (int q = 0; q < 2; ++q) {
              const int r2 = (lane >> 2) + 16 * q;
              const u32x4_t x = *(const u32x4_t*)(slab + o * 2048 + r2 * 64 + ((unit ^ (r2 & 3)) << 4));
              const int rt = wm * C::WTM + mb * 32 + r2;
              if (rt < t.mrows) {
                const int64_t row2 = t.m0 + rt;
                const int f = fb + unit * 8;
                T* dst = o == 2 ? (T*)g.ag + row2 * g.F + f : (T*)g.u + row2 * 2 * g.F + o * g.F + f;
                *(u32x4_t*)dst = x;
              }
            }
          asm volatile("" ::: "memory");  // the reads above before the next writes
        }
        // the row's 32 columns of the block are split between lanes l and l + 32
        part += __shfl_xor(part, 32, 64);
        if (in && lane < 32) g.dgp[row * g.P + fb / 32] = part;
      }
    }
  }
};

// Forward FC2: y[m, n] = sum_f a[m, f] W2[e, n, f].     K = F
template <typename T, class C> struct ProbFC2 {
  typedef ProbFC2 ProbSelf;
  static constexpr bool kEqualTiles = true;  // every tile reduces over the same K
  static constexpr int kRaster = 2;  // preferred tile order (XCD blocks of 8 x 4 tiles)
  static constexpr bool kEpilogueLoads = false;  // the epilogue reads global memory
  typedef KcOp<T, C::BM, C::NW, C::KB, C::DA> OA;
  typedef KcOp<T, C::BN, C::NW, C::KB, C::DB> OB;
  OA A;
  OB B;
  static int grid(const GemmArgs& g) {
    return row_tiles_bound(g.n, g.E, C::BM) * ((ncols(g) + BNU - 1) / BNU);
  }
  static constexpr int BNU = C::BN;  // output columns per tile
  __host__ __device__ static int ncols(const GemmArgs& g) { return g.h; }
  __device__ __forceinline__ bool locate(const GemmArgs& g, Tile& t, int id, int n) const {
    return locate_row_tile<ProbSelf, C::BM, BNU>(g, t, id, n);
  }
  __device__ __forceinline__ bool locate_sub(const GemmArgs& g, Tile& t, int b, int sub) const {
    return locate_row_subtile<ProbSelf, C::BM, BNU>(g, t, b, sub);
  }
  __device__ __forceinline__ static int total_tiles(const GemmArgs& g) {
    return row_tiles<C::BM>(g.offsets, g.E) * ((ncols(g) + BNU - 1) / BNU);
  }
  __device__ __forceinline__ bool active(const GemmArgs& g, const Tile& t, int wm, int wn) const {
    return row_wave_active<ProbSelf, C, BNU>(g, t, wm, wn);
  }
  __host__ __device__ static int reduction(const GemmArgs& g) { return g.F; }
  __device__ __forceinline__ void init(const GemmArgs& g, const Tile& t, int wave, int lane) {
    const uint32_t rowb = (uint32_t)g.F * sizeof(T);
    A.rs = make_rsrc(cptr<T>(g.a, (int64_t)t.m0 * g.F), (int64_t)t.mrows * rowb);
    A.init([&](int r) { return r < t.mrows ? (uint32_t)r * rowb : kOOB; }, wave, lane);
    B.rs = make_rsrc(cptr<T>(g.W2, (int64_t)t.e * g.h * g.F), (int64_t)g.h * rowb);
    B.init([&](int r) { return t.n0 + r < g.h ? (uint32_t)(t.n0 + r) * rowb : kOOB; }, wave, lane);
  }
  __device__ __forceinline__ void init_acc(const GemmArgs&, const Tile&, Accum<C>& acc, int, int,
                                          int) const {
    zero_acc(acc);
  }
  __device__ __forceinline__ void commit(char* As, char* Bs, int wave, int lane) const {
    A.commit(As, wave, lane);
    B.commit(Bs, wave, lane);
  }
  __device__ __forceinline__ void issue(const GemmArgs&, const Tile&, int kt, char* As, char* Bs,
                                        int wave, int) {
    A.issue(As, kt, wave);
    B.issue(Bs, kt, wave);
  }
  __device__ __forceinline__ void epilogue(const GemmArgs& g, const Tile& t, const Accum<C>& acc,
                                           int wm, int wn, int lane, char* slab) const {
    store_rows<T, C>(acc, (T*)g.y, g.h, t, wm, wn, lane, slab);
  }
};

// Router logits: logits[t, e] = sum_k X[t, k] Wr[e, k], stored in fp32.
// FC2's problem with one "expert" holding all T rows: X in `a` (K = h in
// GemmArgs.F), Wr in `W2` (its E_r rows in GemmArgs.h), the logits in `y`.
template <typename T, class C> struct ProbLogits : ProbFC2<T, C> {
  __device__ __forceinline__ void epilogue(const GemmArgs& g, const Tile& t, const Accum<C>& acc,
                                           int wm, int wn, int lane, char*) const {
    store_rows<float, C>(acc, (float*)g.y, g.h, t, wm, wn, lane, nullptr);
  }
};

// Backward FC2 dgrad: dA[m, f] = sum_o dY[tok(m), o] W2[e, o, f]     K = h
// (written to `ag`; the SwiGLU backward happens in the FC1 recomputation).
template <typename T, class C> struct ProbFC2Dgrad {
  typedef ProbFC2Dgrad ProbSelf;
  static constexpr bool kEqualTiles = true;  // every tile reduces over the same K
  static constexpr int kRaster = 2;  // preferred tile order (XCD blocks of 8 x 4 tiles)
  static constexpr bool kEpilogueLoads = false;  // the epilogue reads global memory
  typedef KcOp<T, C::BM, C::NW, C::KB, C::DA> OA;
  typedef KsOp<T, C::BN, C::NW, C::KB, C::DB> OB;
  OA A;
  OB B;
  uint32_t b_ktile;  // bytes of W2 per K tile (BK rows)
  static int grid(const GemmArgs& g) {
    return row_tiles_bound(g.n, g.E, C::BM) * ((ncols(g) + BNU - 1) / BNU);
  }
  static constexpr int BNU = C::BN;  // output columns per tile
  __host__ __device__ static int ncols(const GemmArgs& g) { return g.F; }
  __device__ __forceinline__ bool locate(const GemmArgs& g, Tile& t, int id, int n) const {
    return locate_row_tile<ProbSelf, C::BM, BNU>(g, t, id, n);
  }
  __device__ __forceinline__ bool locate_sub(const GemmArgs& g, Tile& t, int b, int sub) const {
    return locate_row_subtile<ProbSelf, C::BM, BNU>(g, t, b, sub);
  }
  __device__ __forceinline__ static int total_tiles(const GemmArgs& g) {
    return row_tiles<C::BM>(g.offsets, g.E) * ((ncols(g) + BNU - 1) / BNU);
  }
  __device__ __forceinline__ bool active(const GemmArgs& g, const Tile& t, int wm, int wn) const {
    return row_wave_active<ProbSelf, C, BNU>(g, t, wm, wn);
  }
  __host__ __device__ static int reduction(const GemmArgs& g) { return g.h; }
  __device__ __forceinline__ void init(const GemmArgs& g, const Tile& t, int wave, int lane) {
    A.rs = make_rsrc(g.dY, g.T_h_bytes);
    const int32_t* tok = g.tok_of_row + t.m0;
    const uint32_t rowb = (uint32_t)g.h * sizeof(T);
    A.init([&](int r) { return r < t.mrows ? (uint32_t)tok[r] * rowb : kOOB; }, wave, lane);
    const uint32_t ld = (uint32_t)g.F * sizeof(T);  // W2[e] row o holds F values
    B.rs = make_rsrc(cptr<T>(g.W2, (int64_t)t.e * g.h * g.F), (int64_t)g.h * ld);
#pragma clang loop unroll(full)
    for (int i = 0; i < OB::I; ++i) {
      const int col = t.n0 + OB::col_of(i, wave, lane);
      B.voff[i] = col < g.F ? (uint32_t)OB::k_of(i, wave, lane) * ld + col * sizeof(T) : kOOB;
    }
    b_ktile = ld * OB::BKE;
  }
  __device__ __forceinline__ void init_acc(const GemmArgs&, const Tile&, Accum<C>& acc, int, int,
                                          int) const {
    zero_acc(acc);
  }
  __device__ __forceinline__ void commit(char* As, char* Bs, int wave, int lane) const {
    A.commit(As, wave, lane);
    B.commit(Bs, wave, lane);
  }
  __device__ __forceinline__ void issue(const GemmArgs&, const Tile&, int kt, char* As, char* Bs,
                                        int wave, int) {
    A.issue(As, kt, wave);
    B.issue(Bs, kt * b_ktile, wave);
  }
  __device__ __forceinline__ void epilogue(const GemmArgs& g, const Tile& t, const Accum<C>& acc,
                                           int wm, int wn, int lane, char* slab) const {
    store_rows<T, C>(acc, (T*)g.ag, g.F, t, wm, wn, lane, slab);
  }
};

// Router backward's input gradient: dX[t, n] (+)= sum_e D[t, e] Wr[e, n],
// with D the dense dz rows [T, E] (E % 64 == 0).  FC2 dgrad's problem with
// one "expert" of T rows: D in `dY` (K = E in GemmArgs.h, rows through the
// identity `tok_of_row`), Wr in `W2` (h columns in GemmArgs.F), dX in `ag`,
// overwritten or, with `accumulate`, added to in fp32.
template <typename T, class C> struct ProbRouterDx : ProbFC2Dgrad<T, C> {
  // reads dX when accumulating; the epilogue then has kStageSlabBytes of the
  // (idle) stages per wave
  static constexpr bool kEpilogueLoads = true;
  __device__ __forceinline__ void epilogue(const GemmArgs& g, const Tile& t, const Accum<C>& acc,
                                           int wm, int wn, int lane, char* slab) const {
    if (!g.accumulate) {
      store_rows<T, C>(acc, (T*)g.ag, g.F, t, wm, wn, lane, slab);
      return;
    }
    const int ld = g.F;  // % 64 == 0
    if constexpr (sizeof(T) == 2 && C::WTN % 64 == 0 && C::NW * kStageSlabBytes <= C::kLds) {
      // Per 32 rows x 64 columns of the wave's block: the fp32 sums go to the
      // slab (32 rows of 256 bytes, 16-byte units XOR-swizzled by row), then
      // each lane takes 8 consecutive columns of one row, adds the stored
      // bf16 values and writes 16 bytes back: 8 lanes cover one row's 128
      // contiguous bytes.
      const int m0 = __builtin_amdgcn_readfirstlane(t.m0);
      const int mrows = __builtin_amdgcn_readfirstlane(t.mrows);
      const int n0 = __builtin_amdgcn_readfirstlane(t.n0);
      const int rr = lane & 31, half = lane >> 5;
      constexpr int CG = C::WTN / 64;
#pragma clang loop unroll(full)
      for (int mb = 0; mb < C::MB; ++mb)
#pragma clang loop unroll(full)
        for (int cg = 0; cg < CG; ++cg) {
#pragma clang loop unroll(full)
          for (int b = 0; b < 2; ++b)
#pragma clang loop unroll(full)
            for (int gq = 0; gq < 4; ++gq) {
              float v[4];
              acc_run(acc.v[mb][cg * 2 + b], gq, v);
              const int unit = b * 8 + gq * 2 + half;  // 4 fp32 columns
              *(f32x4_t*)(slab + rr * 256 + ((unit ^ (rr & 15)) << 4)) =
                  (f32x4_t){v[0], v[1], v[2], v[3]};
            }
          asm volatile("" ::: "memory");  // the writes above before the reads below
          const int u8 = lane & 7;         // 8-column group of the row
#pragma clang loop unroll(full)
          for (int q = 0; q < 4; ++q) {
            const int r = (lane >> 3) + 8 * q;
            const f32x4_t lo = *(const f32x4_t*)(slab + r * 256 + (((2 * u8) ^ (r & 15)) << 4));
            const f32x4_t hi = *(const f32x4_t*)(slab + r * 256 + (((2 * u8 + 1) ^ (r & 15)) << 4));
            const int row = wm * C::WTM + mb * 32 + r;
            const int col = n0 + wn * C::WTN + cg * 64 + u8 * 8;
            if (row < mrows && col < ld) {
              u32x4_t* o = (u32x4_t*)((T*)g.ag + (int64_t)(m0 + row) * ld + col);
              float f[8];
              unpack16(*o, f, (T*)nullptr);
#pragma clang loop unroll(full)
              for (int c = 0; c < 4; ++c) {
                f[c] += lo[c];
                f[4 + c] += hi[c];
              }
              *o = pack16(f, (T*)nullptr);
            }
          }
          asm volatile("" ::: "memory");  // the reads above before the next writes
        }
      return;
    }
#pragma clang loop unroll(full)
    for (int mb = 0; mb < C::MB; ++mb) {
      const int r = acc_row<C>(wm, mb, lane);
      if (r >= t.mrows) continue;
      T* o = (T*)g.ag + (int64_t)(t.m0 + r) * ld;
#pragma clang loop unroll(full)
      for (int nb = 0; nb < C::NB; ++nb)
#pragma clang loop unroll(full)
        for (int gq = 0; gq < 4; ++gq) {
          const int n = t.n0 + acc_col<C>(wn, nb, gq, lane);
          if (n >= ld) continue;
          float v[4], old[4];
          acc_run(acc.v[mb][nb], gq, v);
          Vec4<T>::unpack(Vec4<T>::load_raw(o + n), old);
#pragma clang loop unroll(full)
          for (int c = 0; c < 4; ++c) v[c] = old[c] + v[c];
          Vec4<T>::store(o + n, v);
        }
    }
  }
};

// Backward FC1 dgrad: dxp[m, n] = sum_c du[m, c] W1[e, c, n].    K = 2F
template <typename T, class C> struct ProbFC1Dgrad {
  typedef ProbFC1Dgrad ProbSelf;
  static constexpr bool kEqualTiles = true;  // every tile reduces over the same K
  static constexpr int kRaster = 2;  // preferred tile order (XCD blocks of 8 x 4 tiles)
  static constexpr bool kEpilogueLoads = false;  // the epilogue reads global memory
  typedef KcOp<T, C::BM, C::NW, C::KB, C::DA> OA;
  typedef KsOp<T, C::BN, C::NW, C::KB, C::DB> OB;
  OA A;
  OB B;
  uint32_t b_ktile;
  static int grid(const GemmArgs& g) {
    return row_tiles_bound(g.n, g.E, C::BM) * ((ncols(g) + BNU - 1) / BNU);
  }
  static constexpr int BNU = C::BN;  // output columns per tile
  __host__ __device__ static int ncols(const GemmArgs& g) { return g.h; }
  __device__ __forceinline__ bool locate(const GemmArgs& g, Tile& t, int id, int n) const {
    return locate_row_tile<ProbSelf, C::BM, BNU>(g, t, id, n);
  }
  __device__ __forceinline__ bool locate_sub(const GemmArgs& g, Tile& t, int b, int sub) const {
    return locate_row_subtile<ProbSelf, C::BM, BNU>(g, t, b, sub);
  }
  __device__ __forceinline__ static int total_tiles(const GemmArgs& g) {
    return row_tiles<C::BM>(g.offsets, g.E) * ((ncols(g) + BNU - 1) / BNU);
  }
  __device__ __forceinline__ bool active(const GemmArgs& g, const Tile& t, int wm, int wn) const {
    return row_wave_active<ProbSelf, C, BNU>(g, t, wm, wn);
  }
  __host__ __device__ static int reduction(const GemmArgs& g) { return 2 * g.F; }
  __device__ __forceinline__ void init(const GemmArgs& g, const Tile& t, int wave, int lane) {
    const uint32_t rowb = (uint32_t)2 * g.F * sizeof(T);
    A.rs = make_rsrc(cptr<T>(g.u, (int64_t)t.m0 * 2 * g.F), (int64_t)t.mrows * rowb);
    A.init([&](int r) { return r < t.mrows ? (uint32_t)r * rowb : kOOB; }, wave, lane);
    const uint32_t ld = (uint32_t)g.h * sizeof(T);  // W1[e] row c holds h values
    B.rs = make_rsrc(cptr<T>(g.W1, (int64_t)t.e * 2 * g.F * g.h), (int64_t)2 * g.F * ld);
#pragma clang loop unroll(full)
    for (int i = 0; i < OB::I; ++i) {
      const int col = t.n0 + OB::col_of(i, wave, lane);
      B.voff[i] = col < g.h ? (uint32_t)OB::k_of(i, wave, lane) * ld + col * sizeof(T) : kOOB;
    }
    b_ktile = ld * OB::BKE;
  }
  __device__ __forceinline__ void init_acc(const GemmArgs&, const Tile&, Accum<C>& acc, int, int,
                                          int) const {
    zero_acc(acc);
  }
  __device__ __forceinline__ void commit(char* As, char* Bs, int wave, int lane) const {
    A.commit(As, wave, lane);
    B.commit(Bs, wave, lane);
  }
  __device__ __forceinline__ void issue(const GemmArgs&, const Tile&, int kt, char* As, char* Bs,
                                        int wave, int) {
    A.issue(As, kt, wave);
    B.issue(Bs, kt * b_ktile, wave);
  }
  __device__ __forceinline__ void epilogue(const GemmArgs& g, const Tile& t, const Accum<C>& acc,
                                           int wm, int wn, int lane, char* slab) const {
    store_rows<T, C>(acc, (T*)g.dxp, g.h, t, wm, wn, lane, slab);
  }
};

// Weight gradients.  Expert e's rows [r0, r0 + K) are the reduction axis:
//   FC2: dW2[e, m, n] (+)= sum_r dY[tok(r), m] * ag[r, n]     M = h,  N = F
//   FC1: dW1[e, m, n] (+)= sum_r du[r, m] * X[tok(r), n]      M = 2F, N = h
// Both operands are K-strided; the token-gathered one (dY for FC2, X for FC1)
// computes its per-lane row offsets for every K tile from the row -> token
// table, one tile ahead.  Tiles (rank, mt, nt) visit experts in descending
// row count.
// kAcc: 1 adds to dW, 0 overwrites it, -1 reads which from GemmArgs (a
// fixed mode lets the compiler drop the other path's loads and their waits).
template <typename T, class C, bool kFC1, int kAcc = -1> struct ProbWgrad {
  static constexpr int kRaster = 0;  // preferred tile order: tile ids in order (no XCD blocks)
  static constexpr bool kEqualTiles = false;  // K = the expert's rows
  static constexpr bool kEpilogueLoads = false;  // no stage slab; the next tile's copies
  // go out before the epilogue (its loads of the old dW, when adding, then wait behind them)
  typedef KsOp<T, C::BM, C::NW, C::KB, C::DA> OA;
  typedef KsOp<T, C::BN, C::NW, C::KB, C::DB> OB;
  static constexpr int IG = kFC1 ? OB::I : OA::I;  // copy instructions of the gathered operand
  OA A;
  OB B;
  static constexpr int D = C::S - 1;              // token prefetch distance (K tiles)
  uint32_t colb[IG];         // gathered operand: byte of this lane's column in a row
  int32_t tok[D][IG];        // gathered operand: tokens of the next D K tiles' rows
  // Per tile, uniform (scalar registers): the expert's row -> token entries,
  // the first of its rows in the non-gathered operand, and its row count.
  // Built once in init, so that a K step's copy issue is a few scalar adds.
  __amdgpu_buffer_rsrc_t trs;
  const char* pbase;
  int Ku;
  __host__ __device__ static int M(const GemmArgs& g) { return kFC1 ? 2 * g.F : g.h; }
  __host__ __device__ static int N(const GemmArgs& g) { return kFC1 ? g.h : g.F; }
  // add into dW for tile t: fixed by the instance (kAcc 0 or 1), else per
  // expert (g.wmode) or per launch (g.accumulate), set by expert_of
  __device__ __forceinline__ bool acc_of(const Tile& t) const {
    return kAcc < 0 ? t.acc != 0 : kAcc == 1;
  }
  static constexpr bool kAccLoads = kAcc != 0 && !kDwAddInEpilogue;
  __host__ __device__ static int tiles_per_expert(const GemmArgs& g) {
    return ((M(g) + C::BM - 1) / C::BM) * ((N(g) + C::BN - 1) / C::BN);
  }
  static int grid(const GemmArgs& g) { return g.E * tiles_per_expert(g); }
  // experts with tiles in this launch: with per-expert modes, the first
  // *g.wexperts of g.order (the others have no rows in the chunk)
  __device__ __forceinline__ static int tile_experts(const GemmArgs& g) {
    if constexpr (kAcc >= 0) return g.E;  // (instances without per-expert modes)
    else return g.wmode != nullptr ? __builtin_amdgcn_readfirstlane(*g.wexperts) : g.E;
  }
  __device__ __forceinline__ static int total_tiles(const GemmArgs& g) {
    return tile_experts(g) * tiles_per_expert(g);
  }
  // does wave (wm, wn) own any element of the tile?
  __device__ __forceinline__ bool active(const GemmArgs& g, const Tile& t, int wm, int wn) const {
    return wm * C::WTM < t.mrows && t.n0 + wn * C::WTN < N(g);
  }
  __device__ __forceinline__ bool expert_of(const GemmArgs& g, Tile& t, int rank) const {
    t.e = g.order[rank];
    t.r0 = g.offsets[t.e];
    t.K = g.offsets[t.e + 1] - t.r0;
    if constexpr (kAcc < 0) {
      const int m = g.wmode != nullptr ? g.wmode[t.e] : (g.accumulate != 0 ? 2 : 1);
      if (m == 0) return false;
      t.acc = m == 2;
    }
    return !(t.K == 0 && acc_of(t));  // nothing to add
  }
  // logical tile L: expert rank L / per (experts in descending row count),
  // then the tile of that expert's grid in raster order
  __device__ __forceinline__ bool locate(const GemmArgs& g, Tile& t, int id, int n) const {
    const int mtn = (M(g) + C::BM - 1) / C::BM, ntn = (N(g) + C::BN - 1) / C::BN;
    const int per = mtn * ntn;
    const int L = logical_of(g.raster, id, n);
    const int rank = L / per;
    if (rank >= tile_experts(g)) return false;
    int mt, nt;
    logical_coords(g.raster, L - rank * per, mtn, ntn, mt, nt);
    if (!expert_of(g, t, rank)) return false;
    t.m0 = mt * C::BM;
    t.n0 = nt * C::BN;
    t.mrows = min(C::BM, M(g) - t.m0);
    return true;
  }
  // quarter `sub` (2 x 2) of logical tile b of the grid with twice the tile
  // size: the split tail of a launch
  __device__ __forceinline__ bool locate_sub(const GemmArgs& g, Tile& t, int b, int sub) const {
    const int mtn2 = (M(g) + 2 * C::BM - 1) / (2 * C::BM), ntn2 = (N(g) + 2 * C::BN - 1) / (2 * C::BN);
    const int per2 = mtn2 * ntn2;
    const int rank = b / per2;
    if (rank >= tile_experts(g)) return false;
    int mt, nt;
    logical_coords(g.raster, b - rank * per2, mtn2, ntn2, mt, nt);
    if (!expert_of(g, t, rank)) return false;
    t.m0 = (2 * mt + (sub >> 1)) * C::BM;
    t.n0 = (2 * nt + (sub & 1)) * C::BN;
    t.mrows = min(C::BM, M(g) - t.m0);
    return t.mrows > 0 && t.n0 < N(g);
  }
  // row k (within the expert) of this lane's copy instruction i in K tile kt
  __device__ __forceinline__ static int k_row(int kt, int i, int wave, int lane) {
    return kt * OA::BKE + (kFC1 ? OB::k_of(i, wave, lane) : OA::k_of(i, wave, lane));
  }
  // Tokens of K tile kt's rows for this lane's copy instructions.  Buffer
  // loads over the expert's rows: the lane's offset is fixed and the K tile
  // goes in the scalar offset, so no address register is rewritten in the K
  // loop (a fragment read reusing one while a load still reads it would have
  // to wait for the load and, vector-memory instructions retiring in order,
  // for every copy in flight); rows past K read as 0 and are masked when the
  // copies are issued.  The values are not touched here, for the same
  // reason.
  __device__ __forceinline__ void load_tokens(int kt, int wave, int lane, int32_t (&dst)[IG]) {
#pragma clang loop unroll(full)
    for (int i = 0; i < IG; ++i)
      dst[i] = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(
          trs, (uint32_t)k_row(0, i, wave, lane) * 4, (uint32_t)kt * OA::BKE * 4, 0);
  }
  // The non-gathered operand (rows r0 .. r0+K of u for FC1, of ag for FC2)
  // gets a resource per K tile, based at the tile's first row, so offsets
  // stay small for any row count and the range ends at the expert's last
  // row (the rows of a last partial K tile past it read as 0).  The range
  // is below 2^31 bytes: 64 rows of at most 2^25 bytes (the shape check
  // bounds one expert's weight, 2 F h elements, below 2^31 bytes, h >= 64).
  __device__ __forceinline__ int ldp(const GemmArgs& g) const { return kFC1 ? 2 * g.F : g.F; }
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t plain_rsrc(const GemmArgs& g, int kt) const {
    const uint32_t ldpb = (uint32_t)ldp(g) * sizeof(T);
    const int k0 = kt * OA::BKE;
    const int rows = min(OA::BKE, Ku - k0);
    return make_rsrc32(pbase + (int64_t)k0 * ldpb, (uint32_t)rows * ldpb);
  }
  __device__ __forceinline__ void init(const GemmArgs& g, const Tile& t, int wave, int lane) {
    const uint32_t ldpb = (uint32_t)ldp(g) * sizeof(T);
    // the tile is the workgroup's: its fields are uniform, which the compiler
    // cannot always prove (the resources must sit in scalar registers)
    const int r0 = __builtin_amdgcn_readfirstlane(t.r0);
    Ku = __builtin_amdgcn_readfirstlane(t.K);
    trs = make_rsrc(g.tok_of_row + r0, (int64_t)max(Ku, 0) * 4);
    pbase = cptr<T>(kFC1 ? g.u : g.ag, (int64_t)r0 * ldp(g));
    const int pcol0 = kFC1 ? t.m0 : t.n0;
    const int plim = kFC1 ? M(g) : N(g);
    const __amdgpu_buffer_rsrc_t grs = make_rsrc(kFC1 ? g.X : g.dY, g.T_h_bytes);
    const int gcol0 = kFC1 ? t.n0 : t.m0;
    const int glim = kFC1 ? N(g) : M(g);
    if (kFC1) {
      B.rs = grs;
#pragma clang loop unroll(full)
      for (int i = 0; i < OA::I; ++i) {
        const int col = pcol0 + OA::col_of(i, wave, lane);
        A.voff[i] = col < plim ? (uint32_t)OA::k_of(i, wave, lane) * ldpb + col * sizeof(T) : kOOB;
      }
#pragma clang loop unroll(full)
      for (int i = 0; i < IG; ++i) {
        const int col = gcol0 + OB::col_of(i, wave, lane);
        colb[i] = col < glim ? col * sizeof(T) : kOOB;
      }
    } else {
      A.rs = grs;
#pragma clang loop unroll(full)
      for (int i = 0; i < OB::I; ++i) {
        const int col = pcol0 + OB::col_of(i, wave, lane);
        B.voff[i] = col < plim ? (uint32_t)OB::k_of(i, wave, lane) * ldpb + col * sizeof(T) : kOOB;
      }
#pragma clang loop unroll(full)
      for (int i = 0; i < IG; ++i) {
        const int col = gcol0 + OA::col_of(i, wave, lane);
        colb[i] = col < glim ? col * sizeof(T) : kOOB;
      }
    }
#pragma clang loop unroll(full)
    for (int d = 0; d < D; ++d) load_tokens(d, wave, lane, tok[d]);
  }
  // Accumulating into dW: by default the accumulators start at zero and the
  // epilogue adds the old dW values (dW = old + this launch's sum).  Built
  // with MEMFINE_DW_ADD_IN_EPILOGUE=0 they start from the old values instead,
  // loaded with the tile's first operand copies.  Rows past the tile and runs
  // past N load from clamped in-range addresses; those accumulators are
  // never stored.
  __device__ __forceinline__ void init_acc(const GemmArgs& g, const Tile& t, Accum<C>& acc, int wm,
                                          int wn, int lane) const {
    if (kDwAddInEpilogue || !acc_of(t)) {
      zero_acc(acc);
      return;
    }
    const float* dW = (kFC1 ? g.dW1 : g.dW2) + (int64_t)t.e * M(g) * N(g);
    const int Nn = N(g);
#pragma clang loop unroll(full)
    for (int mb = 0; mb < C::MB; ++mb) {
      const int r = acc_row<C>(wm, mb, lane);
      const float* o = dW + (int64_t)(t.m0 + (r < t.mrows ? r : 0)) * Nn;
#pragma clang loop unroll(full)
      for (int nb = 0; nb < C::NB; ++nb)
#pragma clang loop unroll(full)
        for (int gq = 0; gq < 4; ++gq) {
          const int n = t.n0 + acc_col<C>(wn, nb, gq, lane);
          const f32x4_t v = Vec4<float>::load_raw(o + (n < Nn ? n : t.n0));
#pragma clang loop unroll(full)
          for (int c = 0; c < 4; ++c) acc.v[mb][nb][gq * 4 + c] = v[c];
        }
    }
  }
  __device__ __forceinline__ void commit(char* As, char* Bs, int wave, int lane) const {
    A.commit(As, wave, lane);
    B.commit(Bs, wave, lane);
  }
  // byte offsets of the gathered operand's copies of K tile kt (tokens in tok[0])
  __device__ __forceinline__ void gather_offsets(const GemmArgs& g, int kt, int wave, int lane,
                                                 uint32_t (&gv)[IG]) const {
    const uint32_t rowb = (uint32_t)g.h * sizeof(T);
    if ((kt + 1) * OA::BKE <= Ku) {
      // a whole K tile of the expert's rows (every tile but a partial last one)
#pragma clang loop unroll(full)
      for (int i = 0; i < IG; ++i) gv[i] = (uint32_t)tok[0][i] * rowb + colb[i];
    } else {
      // branch-free: a row past K or a column past the operand gets bit 31
      // (kOOB), which puts the offset past the resource (a byte of X or dY is
      // below 2^31); colb already is kOOB for such a column
#pragma clang loop unroll(full)
      for (int i = 0; i < IG; ++i)
        gv[i] = ((uint32_t)tok[0][i] * rowb + colb[i]) |
                (k_row(kt, i, wave, lane) >= Ku ? kOOB : 0u);
    }
  }
  __device__ __forceinline__ void issue(const GemmArgs& g, const Tile& t, int kt, char* As,
                                        char* Bs, int wave, int lane) {
    if constexpr (kFC1) gather_offsets(g, kt, wave, lane, B.voff);
    else gather_offsets(g, kt, wave, lane, A.voff);
    if (kFC1) A.rs = plain_rsrc(g, kt);
    else B.rs = plain_rsrc(g, kt);
    A.issue(As, 0, wave);
    B.issue(Bs, 0, wave);
#pragma clang loop unroll(full)
    for (int d = 0; d + 1 < D; ++d)
#pragma clang loop unroll(full)
      for (int i = 0; i < IG; ++i) tok[d][i] = tok[d + 1][i];
    load_tokens(kt + D, wave, lane, tok[D - 1]);  // D tiles ahead
  }
  // Vector-memory stores epilogue() issues: every one, whatever the tile's
  // extent (elements outside it get an offset past the range).  When it adds
  // into dW it also loads the old values and waits for them, so the loads
  // are retired, with everything issued before them, when it returns.
  static constexpr int kEpiStores = C::MB * C::NB * 4;
  __device__ __forceinline__ void epilogue(const GemmArgs& g, const Tile& t, const Accum<C>& acc,
                                           int wm, int wn, int lane, char* slab) const {
    const int Nn = N(g);  // % 64 == 0: a run of 4 columns is all in or all out
    const uint32_t rowb = (uint32_t)Nn * sizeof(float);
    // the tile is the workgroup's: its fields are uniform, which the compiler
    // cannot always prove (the resource must sit in scalar registers)
    const int e = __builtin_amdgcn_readfirstlane(t.e);
    const int m0 = __builtin_amdgcn_readfirstlane(t.m0);
    const int mrows = __builtin_amdgcn_readfirstlane(t.mrows);
    const __amdgpu_buffer_rsrc_t rs =
        make_rsrc((kFC1 ? g.dW1 : g.dW2) + (int64_t)e * M(g) * Nn + (int64_t)m0 * Nn,
                  (int64_t)mrows * rowb);
    const bool add = kDwAddInEpilogue && acc_of(t);
#pragma clang loop unroll(full)
    for (int mb = 0; mb < C::MB; ++mb) {
      const int r = acc_row<C>(wm, mb, lane);
      const uint32_t ro = r < mrows ? (uint32_t)r * rowb : kOOB;
      f32x4_t old[C::NB][4];
      if (add) {
#pragma clang loop unroll(full)
        for (int nb = 0; nb < C::NB; ++nb)
#pragma clang loop unroll(full)
          for (int gq = 0; gq < 4; ++gq) {
            const int n = t.n0 + acc_col<C>(wn, nb, gq, lane);
            old[nb][gq] = __builtin_bit_cast(
                f32x4_t, load_reg16(rs, n < Nn ? ro + (uint32_t)n * sizeof(float) : kOOB, 0));
          }
      }
#pragma clang loop unroll(full)
      for (int nb = 0; nb < C::NB; ++nb)
#pragma clang loop unroll(full)
        for (int gq = 0; gq < 4; ++gq) {
          const int n = t.n0 + acc_col<C>(wn, nb, gq, lane);
          float v[4];
          acc_run(acc.v[mb][nb], gq, v);
          if (add)
#pragma clang loop unroll(full)
            for (int c = 0; c < 4; ++c) v[c] += old[nb][gq][c];
          store_f32x4(rs, n < Nn ? ro + (uint32_t)n * sizeof(float) : kOOB, v);
        }
    }
  }
};

// ------------------------------------------------------------------ kernel
// s_waitcnt vmcnt(N): at most N vector-memory loads of this wave in flight
template <int N> __device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt is a 6-bit counter");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// K loop over an S-stage ring of LDS tiles.  Tile kt+S-1 is copied into the
// stage that held tile kt-1 while the waves multiply tile kt.  Before tile
// kt is used, each wave waits until only the copies of the tiles issued
// after it may still be in flight (loads retire in order), then a barrier
// publishes every wave's copies and also certifies that all waves are done
// with tile kt-1, whose stage the next copy overwrites.
struct NoNext {
  __device__ __forceinline__ void operator()(char*, int, int) const {}
};
// Problems whose init_acc may load the accumulators (P::acc_on tells when).
template <class P, class = void> struct AccLoads { static constexpr bool value = false; };
template <class P> struct AccLoads<P, decltype((void)P::kAccLoads)> {
  static constexpr bool value = P::kAccLoads;
};
// Problems whose epilogue leaves at most P::kEpiStores vector-memory
// instructions in flight (its stores; loads it waits for) can take the deep
// prefetch below.
template <class P, class = void> struct HasEpiStores { static constexpr bool value = false; };
template <class P> struct HasEpiStores<P, decltype((void)P::kEpiStores)> {
  static constexpr bool value = true;
};
template <class C, class P>
constexpr bool kDeep = C::DIRECT && C::S == 2 && HasEpiStores<P>::value;
// K tiles of a tile's reduction.
template <typename T, class C> __device__ __forceinline__ int k_tiles(const Tile& t) {
  constexpr int BKE = C::KB / (int)sizeof(T);
  return (t.K + BKE - 1) / BKE;
}
// Copies of a located tile's first S - 1 K tiles (direct copies only).
template <typename T, class C, class P>
__device__ __forceinline__ void issue_prologue(const GemmArgs& g, char* smem, P& p, const Tile& t,
                                               int w, int lane) {
  const int nk = k_tiles<T, C>(t);
#pragma clang loop unroll(full)
  for (int j = 0; j < C::S - 1; ++j) {
    char* st = smem + j * C::kStage;
    if (j < nk) p.issue(g, t, j, st, st + C::BM * C::KB, w, lane);
  }
}

// Copies of a located tile's first two K tiles into both stages of a
// two-stage ring, issued before the previous tile's epilogue: its stores then
// queue behind them and the first two K steps need not wait for the stores.
template <typename T, class C, class P>
__device__ __forceinline__ void issue_prologue2(const GemmArgs& g, char* smem, P& p, const Tile& t,
                                                int w, int lane) {
  static_assert(C::DIRECT && C::S == 2, "two-stage direct-copy ring");
  const int nk = k_tiles<T, C>(t);
#pragma clang loop unroll(full)
  for (int j = 0; j < 2; ++j) {
    char* st = smem + j * C::kStage;
    if (j < nk) p.issue(g, t, j, st, st + C::BM * C::KB, w, lane);
  }
}
// vmcnt operand for "the N most recent vector-memory instructions may still
// be in flight"; with more than the counter holds in flight, waiting for 62
// still retires everything older (the wave cannot have more outstanding)
constexpr int vm_cap(int n) { return n < 62 ? n : 62; }

// One output tile.  `prefetched`: the previous tile of this workgroup already
// ran p.init and issued the copies of the first S - 1 K tiles.  `next` runs
// after the K loop, before the epilogue (with the LDS stages free once it
// has passed a barrier).
//
// `deep` (two-stage direct-copy rings of problems whose epilogue leaves at
// most P::kEpiStores vector-memory instructions in flight): the previous tile
// issued this tile's first two K tiles (issue_prologue2) and then its
// epilogue, so at K step 0 the copies of K tile 1 and those stores, and at
// step 1 the stores, were issued after the copies waited for.  Vector-memory
// instructions retire in order, so waiting until only that many are in
// flight suffices, and the stores drain under the first two K steps.
template <typename T, class C, class P, int kArray = 0, class Next = NoNext>
__device__ __forceinline__ void run_located(const GemmArgs& g, char* smem, P& p, const Tile& t,
                                            bool prefetched = false, Next next = Next(),
                                            bool deep = false) {
  const int lane = threadIdx.x & 63;
  // the wave index in a scalar register: every LDS destination of a copy
  // (M0) and every per-wave choice below is then scalar arithmetic, with no
  // VGPR address and readfirstlane per copy instruction
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int wm, wn;
  C::wave_role(w, wm, wn);
  // a wave whose whole block lies past the tile's rows or columns skips its
  // fragment reads and MFMAs (its epilogue stores nothing)
  const bool active = p.active(g, t, wm, wn);
  if (!prefetched) p.init(g, t, w, lane);
  Accum<C> acc;
  p.init_acc(g, t, acc, wm, wn, lane);
  // Accumulators loaded from memory: wait here, once.  Left to the compiler,
  // the waits for them land inside the K loop's multiply (its loop state
  // merges this entry with the loop's own), where they also wait for the
  // copies each K step has just issued.
  if constexpr (AccLoads<P>::value)
    if (p.acc_of(t)) wait_vm<0>();
  constexpr int kCopies = P::OA::I + P::OB::I;  // copy instructions per wave per K tile
  const int nk = k_tiles<T, C>(t);
  if constexpr (C::DIRECT) {
    if (!prefetched) issue_prologue<T, C, P>(g, smem, p, t, w, lane);
    FragSets<T, C> fr;
    for (int kt = 0; kt < nk; ++kt) {
      if constexpr (kDirectPrio == 1) __builtin_amdgcn_s_setprio(2);
      if constexpr (kDeep<C, P>) {
        if (deep && kt == 0 && nk > 1) wait_vm<vm_cap(kCopies + P::kEpiStores)>();
        else if (deep && kt < 2) wait_vm<vm_cap(P::kEpiStores)>();
        else wait_vm<0>();
      } else if (kt + C::S - 2 < nk) {
        wait_vm<(C::S - 2) * kCopies>();
      } else {
        wait_vm<0>();
      }
      // A bare s_barrier: __syncthreads() would add a memory fence, for which
      // the compiler waits for every copy in flight (vmcnt(0)) and so defeats
      // the deeper stages.  The explicit wait above already makes this wave's
      // copies of tile kt visible.  Every LDS read of the stage the next copy
      // overwrites has returned: its MFMA has issued, or, for the step carried
      // over the barrier (kCarryStep), the reads are waited for here.
      if constexpr (kCarryStep) wait_lgkm0();
      __builtin_amdgcn_s_barrier();
      if (kt + C::S - 1 < nk && !(deep && kt + C::S - 1 < 2)) {
        char* st = smem + ((kt + C::S - 1) % C::S) * C::kStage;
        p.issue(g, t, kt + C::S - 1, st, st + C::BM * C::KB, w, lane);
      }
      if constexpr (kDirectPrio == 1) __builtin_amdgcn_s_setprio(0);
      char* cur = smem + (kt % C::S) * C::kStage;
      if constexpr (kCarryStep) {
        if (active) {
          if (kt == 0)
            mma_tile_carry<T, C, typename P::OA, typename P::OB, false>(cur, cur + C::BM * C::KB, acc,
                                                                     wm, wn, lane, fr);
          else
            mma_tile_carry<T, C, typename P::OA, typename P::OB, true>(cur, cur + C::BM * C::KB, acc,
                                                                    wm, wn, lane, fr);
        }
      } else {
        if (active)
          mma_tile<T, C, typename P::OA, typename P::OB>(cur, cur + C::BM * C::KB, acc, wm, wn, lane);
      }
    }
    if constexpr (kCarryStep)
      if (active && nk > 0) mma_flush<T, C>(acc, fr);
  } else {
    // Register-staged double buffer: the loads of tile kt + 1 are in flight
    // while tile kt is multiplied, then written to the stage that tile kt - 1
    // used (free since the barrier that opened this step).
    static_assert(C::S == 2, "register staging uses two LDS stages");
    if (nk > 0) {
      p.issue(g, t, 0, smem, smem + C::BM * C::KB, w, lane);
      wait_vm<0>();
      p.commit(smem, smem + C::BM * C::KB, w, lane);
    }
    FragSets<T, C> fr;
    for (int kt = 0; kt < nk; ++kt) {
      // (the fence of __syncthreads also waits for the carried step's reads)
      __syncthreads();
      char* cur = smem + (kt & 1) * C::kStage;
      char* nxt = smem + ((kt + 1) & 1) * C::kStage;
      const bool more = kt + 1 < nk;
      if (more) p.issue(g, t, kt + 1, nxt, nxt + C::BM * C::KB, w, lane);
      if constexpr (kCarryStep) {
        if (active) {
          if (kt == 0)
            mma_tile_carry<T, C, typename P::OA, typename P::OB, false>(cur, cur + C::BM * C::KB, acc,
                                                                     wm, wn, lane, fr);
          else
            mma_tile_carry<T, C, typename P::OA, typename P::OB, true>(cur, cur + C::BM * C::KB, acc,
                                                                    wm, wn, lane, fr);
        }
      } else {
        if (active)
          mma_tile<T, C, typename P::OA, typename P::OB>(cur, cur + C::BM * C::KB, acc, wm, wn, lane);
      }
      if (more) {
        wait_vm<0>();
        p.commit(nxt, nxt + C::BM * C::KB, w, lane);
      }
    }
    if constexpr (kCarryStep)
      if (active && nk > 0) mma_flush<T, C>(acc, fr);
  }
  next(smem, w, lane);
  char* slab = slab_of<C, kArray>(smem, w);
  if constexpr (P::kEpilogueLoads && C::NW * kStageSlabBytes <= C::kLds) {
    // No copies of a next tile are in flight during such an epilogue (they
    // are issued after it): once every wave is past its last multiply, the
    // stages are free and each wave takes kStageSlabBytes of them.
    __syncthreads();
    slab = smem + w * kStageSlabBytes;
  }
  p.epilogue(g, t, acc, wm, wn, lane, slab);
}

template <typename T, class C, class P>
__device__ __forceinline__ void run_tile(const GemmArgs& g, char* smem, int id, int n) {
  P p;
  Tile t;
  if (p.locate(g, t, id, n)) run_located<T, C, P>(g, smem, p, t);
}

template <typename T, class C, class P>
__global__ __launch_bounds__(C::kThreads, C::kMinWaves)
__attribute__((amdgpu_waves_per_eu(C::kMinWaves, C::kMinWaves))) void grouped_gemm_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(1024))) char smem[C::kLds + kSlabArea<C>];
  const int n = min((int)gridDim.x, P::total_tiles(g));
  if ((int)blockIdx.x < n) run_tile<T, C, P>(g, smem, blockIdx.x, n);
}

// Launches of direct-copy tiles of equal cost run persistent: one workgroup
// per CU walks ids blockIdx.x, + cus, ..., with the next tile's first copies
// in flight during the epilogue (after it, where the epilogue loads).  The
// others run one tile per workgroup: register-staged copies (a launch
// option) leave no registers to carry a next tile, and weight-gradient tiles
// (K = the expert's rows) differ in cost, which the hardware's dynamic
// dispatch balances better than a fixed stride (measured 3-8 % faster).
template <class C, class P>
constexpr bool kPersistent = C::DIRECT && C::S == 2 && P::kEqualTiles;
// Weight gradients (direct copies, tile cost = the expert's rows) run
// persistent with a tile counter when the launch provides one: each
// workgroup takes the next tile in launch order (experts by descending row
// count) from the counter, fetched one tile ahead, so that CUs that finish
// early take more tiles; the next tile's first copies fly during the
// epilogue's dW stores.
template <class C, class P>
constexpr bool kDynamic = C::DIRECT && C::S == 2 && !P::kEqualTiles && !P::kEpilogueLoads;

// A launch with a split tail.  Tiles of configuration C fill the full
// rounds (floor(tiles / cus) * cus of them); when the last, partial round
// would hold at most cus / 2 tiles, each of its tiles runs instead as four
// quarter tiles of configuration CQ (same workgroup size), spread over four
// times as many CUs, so the launch ends about three quarters of a round
// earlier.  A row-grouped tile count depends on the chunk's expert offsets
// and is computed here.  (The weight gradients' last round holds the experts
// with the fewest rows.)
template <typename T, class C, class CQ, class P, class PQ>
__global__ __launch_bounds__(C::kThreads, C::kMinWaves)
__attribute__((amdgpu_waves_per_eu(C::kMinWaves, C::kMinWaves))) void grouped_gemm_split_kernel(
    GemmArgs g) {
  static_assert(C::kThreads == CQ::kThreads && C::kLds >= CQ::kLds, "quarter tiles must fit");
  static_assert(CQ::BM * 2 == C::BM && CQ::BN * 2 == C::BN, "quarter tiles of the same grid");
  // One LDS object: the stages, then the epilogue slabs or (dynamic launches,
  // whose epilogues take no slab) the next tile index.
  // With a second __shared__ variable the compiler scopes every LDS access
  // by variable and then cannot tell a fragment read of one stage from the
  // copies into the other, so each K step's reads would wait for the next
  // step's copies.
  constexpr int kArray = C::kLds + (kSlabArea<C> > 16 ? kSlabArea<C> : 16);
  __shared__ __attribute__((aligned(1024))) char smem[kArray];
  const int tiles = P::total_tiles(g);
  const int full = tiles / g.cus * g.cus, rem = tiles - full;
  const bool split = g.split_tail && 2 * rem <= g.cus;
  const int nmain = split ? full : tiles;   // ids that run whole tiles
  const int stride = gridDim.x;
  if constexpr (kPersistent<C, P>) {
    // Whole tiles: ids blockIdx.x, + stride, ...  At the end of each tile's
    // K loop the next tile is located, its copy offsets set and its first K
    // tiles' copies issued, so that they fly while this tile's epilogue runs.
    P p;
    Tile t;
    int id = blockIdx.x;
    bool ok = false;
    while (id < nmain && !(ok = p.locate(g, t, id, nmain))) id += stride;
    bool pre = false;
    while (ok) {
      P pn;
      Tile tn;
      int idn = id + stride;
      bool okn = false;
      // every wave at the hook or past the epilogue is past its last MFMA,
      // so its LDS reads have returned: after a barrier the stages are free
      auto next = [&](char* sm, int w, int lane) {
        while (idn < nmain && !(okn = pn.locate(g, tn, idn, nmain))) idn += stride;
        if (okn) {
          __builtin_amdgcn_s_barrier();
          pn.init(g, tn, w, lane);
          issue_prologue<T, C, P>(g, sm, pn, tn, w, lane);
        }
      };
      if constexpr (!P::kEpilogueLoads) {
        run_located<T, C, P>(g, smem, p, t, pre, next);   // copies fly during the epilogue
      } else {
        // the epilogue's own loads would wait behind earlier copies: issue
        // the next tile's copies once the epilogue is done
        run_located<T, C, P>(g, smem, p, t, pre);
        next(smem, __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), threadIdx.x & 63);
      }
      p = pn;
      t = tn;
      id = idn;
      ok = okn;
      pre = okn;
    }
    if (split) {
      for (int q = blockIdx.x; q < 4 * rem; q += stride) {
        PQ pq;
        Tile tq;
        __syncthreads();  // the previous tile's waves are done with the stages
        if (pq.locate_sub(g, tq, full + q / 4, q % 4)) run_located<T, CQ, PQ, kArray>(g, smem, pq, tq);
      }
    }
  } else if (kDynamic<C, P> && g.tile_ctr != nullptr) {
    // Three LDS words: slot 2 for grab(), slots 0 and 1 for the tile index
    // fetched ahead, alternating from one tile to the next.  A wave reads
    // slot p after the barrier that follows thread 0's write; thread 0 writes
    // slot p again two tiles later, after it has passed the next tile's
    // barrier, which every wave reaches only after its read - even when the
    // tile in between has no K steps (an expert without rows) and so no K-loop
    // barrier.
    int32_t* s_next = reinterpret_cast<int32_t*>(smem + C::kLds);
    // thread 0 takes a tile index; every wave reads it after a barrier (and
    // again before thread 0 may overwrite it)
    auto grab = [&]() {
      if (threadIdx.x == 0) s_next[2] = atomicAdd(g.tile_ctr, 1);
      __syncthreads();
      const int v = __builtin_amdgcn_readfirstlane(s_next[2]);  // uniform: scalar tile state
      __syncthreads();
      return v;
    };
    int par = 0;
    P p;
    Tile t;
    int v = grab();
    bool pre = false;
    for (;;) {
      if (!pre) {
        while (v < nmain && !p.locate(g, t, v, nmain)) v = grab();
        if (v >= nmain) break;
      }
      // thread 0: the next tile index, fetched during this tile.  Left
      // undefined for the other threads (which never read it), so that no
      // copy of the result at the end of the branch waits for the atomic -
      // and, vector-memory instructions retiring in order, for everything
      // issued before it.
      // (The offset is an opaque per-lane zero: with a provably uniform
      // address the compiler aggregates the atomic over the wave and reads
      // its result back at once.)
      int32_t ahead;
      if (threadIdx.x == 0) {
        int32_t zero;
        asm volatile("v_mov_b32 %0, 0" : "=v"(zero));
        ahead = atomicAdd(g.tile_ctr + zero, 1);
      }
      P pn;
      Tile tn;
      int vn = nmain;
      bool okn = false;
      run_located<T, C, P>(g, smem, p, t, pre, [&](char* sm, int w, int lane) {
        if (threadIdx.x == 0) s_next[par] = ahead;
        __syncthreads();  // s_next is visible; every wave is past its last MFMA
        vn = __builtin_amdgcn_readfirstlane(s_next[par]);
        okn = vn < nmain && pn.locate(g, tn, vn, nmain);
        if (okn) {
          pn.init(g, tn, w, lane);
          if constexpr (kDeep<C, P>) issue_prologue2<T, C, P>(g, sm, pn, tn, w, lane);
          else issue_prologue<T, C, P>(g, sm, pn, tn, w, lane);
        }
      }, kDeep<C, P> && pre);
      if (okn) {
        p = pn;
        t = tn;
      }
      v = vn;
      pre = okn;
      par ^= 1;
      // without a prefetched tile, the grab in the locate loop above (or the
      // quarter-tile barrier below) separates this tile's LDS use from the
      // next one's, and lets every wave read s_next before it changes
      if (!okn) __syncthreads();
    }
    if (split) {
      for (int q = blockIdx.x; q < 4 * rem; q += stride) {
        PQ pq;
        Tile tq;
        __syncthreads();  // the previous tile's waves are done with the stages
        if (pq.locate_sub(g, tq, full + q / 4, q % 4)) run_located<T, CQ, PQ, kArray>(g, smem, pq, tq);
      }
    }
  } else {
    // one tile per workgroup
    const int id = blockIdx.x;
    if (id < nmain) {
      P p;
      Tile t;
      if (p.locate(g, t, id, nmain)) run_located<T, C, P>(g, smem, p, t);
    } else if (split && id < full + 4 * rem) {
      PQ p;
      Tile t;
      const int q = id - full;
      if (p.locate_sub(g, t, full + q / 4, q % 4)) run_located<T, CQ, PQ, kArray>(g, smem, p, t);
    }
  }
}

// The dgrad and the wgrad of one FC layer in one launch (nd + nw workgroups;
// the two problems are independent).  Every dgrad tile reduces over the same
// K (h or 2F); a wgrad tile reduces over its expert's rows.  Workgroups are
// dealt longest tile first, as far as that matters: first the wgrad tiles of
// the experts with at least K rows (the wgrad grid already lists experts by
// descending rows), then the dgrad tiles and the remaining, shorter wgrad
// tiles interleaved in proportion (workgroup j of this part runs dgrad tile
// floor(j nd / m) when that value steps at j, else the next wgrad tile).  The
// CUs thus run a mix of both problems: the memory-heavy epilogues of one
// overlap the matrix-core phases of the other, and neither leaves a
// half-empty last round.
template <typename T, class C, class PD, class PW>
__global__ __launch_bounds__(C::kThreads, C::kMinWaves)
__attribute__((amdgpu_waves_per_eu(C::kMinWaves, C::kMinWaves))) void grouped_gemm_bwd_pair_kernel(
    GemmArgs g, int nd, int nw) {
  __shared__ __attribute__((aligned(1024))) char smem[C::kLds + kSlabArea<C>];
  const int Kd = PD::reduction(g);
  // first rank (experts by descending rows) with fewer than Kd rows
  int lo = 0, hi = g.E;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1, e = g.order[mid];
    if (g.offsets[e + 1] - g.offsets[e] >= Kd) lo = mid + 1;
    else hi = mid;
  }
  const int lead = lo * PW::tiles_per_expert(g);
  const int i = blockIdx.x;
  if (i < lead) {
    run_tile<T, C, PW>(g, smem, i, nw);
    return;
  }
  const int64_t j = i - lead, m = (int64_t)nd + (nw - lead);
  const int a = (int)(j * nd / m), b = (int)((j + 1) * nd / m);
  if (b > a) run_tile<T, C, PD>(g, smem, a, nd);
  else run_tile<T, C, PW>(g, smem, lead + (int)(j - a), nw);
}

template <template <typename, class> class PT, class C>
hipError_t launch_cfg(const GemmArgs& g, hipStream_t s) {
  const int blocks = PT<float, C>::grid(g);
  if (blocks <= 0) return hipSuccess;
  if (g.dtype == 0)
    grouped_gemm_kernel<bf16_t, C, PT<bf16_t, C>><<<blocks, C::kThreads, 0, s>>>(g);
  else
    grouped_gemm_kernel<float, Small, PT<float, Small>><<<PT<float, Small>::grid(g), Small::kThreads,
                                                          0, s>>>(g);
  return hipGetLastError();
}

template <template <typename, class> class P1, template <typename, class> class P2, class C>
hipError_t launch_pair_cfg(const GemmArgs& g, hipStream_t s) {
  if (g.dtype != 0) {
    const int n1 = P1<float, Small>::grid(g), n2 = P2<float, Small>::grid(g);
    if (n1 + n2 <= 0) return hipSuccess;
    grouped_gemm_bwd_pair_kernel<float, Small, P1<float, Small>, P2<float, Small>>
        <<<n1 + n2, Small::kThreads, 0, s>>>(g, n1, n2);
  } else {
    const int n1 = P1<bf16_t, C>::grid(g), n2 = P2<bf16_t, C>::grid(g);
    if (n1 + n2 <= 0) return hipSuccess;
    grouped_gemm_bwd_pair_kernel<bf16_t, C, P1<bf16_t, C>, P2<bf16_t, C>>
        <<<n1 + n2, C::kThreads, 0, s>>>(g, n1, n2);
  }
  return hipGetLastError();
}

// Workgroup-rounds a grid of `tiles` tiles takes on the whole chip.
inline double rounds(int tiles, int per_cu) {
  const int slots = 256 * per_cu;
  return (double)((tiles + slots - 1) / slots);
}

using Big8 = Cfg<256, 256, 2, 4, 2>;        // 8 waves of 128 x 64
using Big8R = Cfg<256, 256, 2, 4, 2, 128, 0>;  // Big8 with register-staged copies
using Quarter8 = Cfg<128, 128, 4, 2, 2>;        // quarter tiles of Big8 (8 waves of 32 x 64)

template <typename T, class C> using FC1Fwd = ProbFC1<T, C, false>;
template <typename T, class C> using FC1Bwd = ProbFC1<T, C, true>;
template <typename T, class C> using FC2W = ProbWgrad<T, C, false>;
template <typename T, class C> using FC1W = ProbWgrad<T, C, true>;
template <typename T, class C> using FC2WNew = ProbWgrad<T, C, false, 0>;
template <typename T, class C> using FC2WAdd = ProbWgrad<T, C, false, 1>;
template <typename T, class C> using FC1WNew = ProbWgrad<T, C, true, 0>;
template <typename T, class C> using FC1WAdd = ProbWgrad<T, C, true, 1>;

template <template <typename, class> class PT, class C, class CQ>
hipError_t launch_split_cfg(const GemmArgs& g, hipStream_t s) {
  const int bound = PT<bf16_t, C>::grid(g);
  if (bound <= 0) return hipSuccess;
  const bool dynamic = kDynamic<C, PT<bf16_t, C>> && g.tile_ctr != nullptr;
  if (dynamic) {  // the tile counter starts at 0 for this launch
    const hipError_t err = launch_fill_i32(g.tile_ctr, 1, 0, s);
    if (err != hipSuccess) return err;
  }
  const int blocks = (kPersistent<C, PT<bf16_t, C>> || dynamic) ? std::min(bound, g.cus)
                                                                 : bound + 3 * (g.cus / 2);
  grouped_gemm_split_kernel<bf16_t, C, CQ, PT<bf16_t, C>, PT<bf16_t, CQ>>
      <<<blocks, C::kThreads, 0, s>>>(g);
  return hipGetLastError();
}

// Pick the tile shape.  The 256 x 256 tile on 8 waves (one workgroup per CU,
// two waves per SIMD, 128 x 64 per wave) measured fastest on every workload
// shape here, from 8k to 65k slots and C = 1..4; the 128 x 128 tile (two
// workgroups per CU) only serves grids too small to give most CUs a tile.
// Every problem takes direct copies into LDS: the dgrads (an activation-row
// operand and a K-strided weight operand) and the router's dX measured 2-8 %
// faster with them than with register-staged copies, which remain a launch
// option (MEMFINE_TILE_256_REG).
template <template <typename, class> class PT>
hipError_t launch_auto(const GemmArgs& g_in, hipStream_t s) {
  GemmArgs g = g_in;
  if (g.raster < 0) g.raster = PT<float, Big8>::kRaster;
  if (g.dtype != 0) return launch_cfg<PT, Small>(g, s);
  switch (g.tile_override) {  // memfine_launch_options.tile
    case 1: return launch_cfg<PT, Small>(g, s);
    case 2: return launch_cfg<PT, Big8>(g, s);
    case 3: return launch_cfg<PT, Big8R>(g, s);
    default: break;
  }
  if (PT<float, Big8>::grid(g) >= 128) {
    if (g.split_tail) return launch_split_cfg<PT, Big8, Quarter8>(g, s);
    return launch_cfg<PT, Big8>(g, s);
  }
  return launch_cfg<PT, Small>(g, s);
}

template <template <typename, class> class P1, template <typename, class> class P2>
hipError_t launch_pair(const GemmArgs& g_in, hipStream_t s) {
  GemmArgs g = g_in;
  if (g.raster < 0) g.raster = 0;
  if (g.dtype == 0 && P1<float, Big8>::grid(g) + P2<float, Big8>::grid(g) < 128)
    return launch_pair_cfg<P1, P2, Small>(g, s);
  return launch_pair_cfg<P1, P2, Big8>(g, s);
}


}  // namespace

int dgate_partials(int F) { return (F + 31) / 32; }

hipError_t launch_fc1_fwd(const GemmArgs& g, hipStream_t s) { return launch_auto<FC1Fwd>(g, s); }
hipError_t launch_fc1_recompute(const GemmArgs& g, hipStream_t s) { return launch_auto<FC1Bwd>(g, s); }
hipError_t launch_fc2_fwd(const GemmArgs& g, hipStream_t s) { return launch_auto<ProbFC2>(g, s); }
hipError_t launch_fc2_dgrad(const GemmArgs& g, hipStream_t s) { return launch_auto<ProbFC2Dgrad>(g, s); }
hipError_t launch_fc1_dgrad(const GemmArgs& g, hipStream_t s) { return launch_auto<ProbFC1Dgrad>(g, s); }
hipError_t launch_fc2_wgrad(const GemmArgs& g, hipStream_t s) {
  if (g.wmode != nullptr) return launch_auto<FC2W>(g, s);  // per-expert modes
  return g.accumulate ? launch_auto<FC2WAdd>(g, s) : launch_auto<FC2WNew>(g, s);
}
hipError_t launch_fc1_wgrad(const GemmArgs& g, hipStream_t s) {
  if (g.wmode != nullptr) return launch_auto<FC1W>(g, s);  // per-expert modes
  return g.accumulate ? launch_auto<FC1WAdd>(g, s) : launch_auto<FC1WNew>(g, s);
}
hipError_t launch_router_dx(const GemmArgs& g, hipStream_t s) {
  return launch_auto<ProbRouterDx>(g, s);
}
hipError_t launch_router_logits(const GemmArgs& g, hipStream_t s) {
  return launch_auto<ProbLogits>(g, s);
}
hipError_t launch_fc1_dgrad_wgrad(const GemmArgs& g, hipStream_t s) {
  return launch_pair<ProbFC1Dgrad, FC1W>(g, s);
}

}  // namespace memfine
