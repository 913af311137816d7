// Grouped expert GEMMs of the chunked MoE layer on gfx950 matrix cores.
//
// Every GEMM of the expert SwiGLU FFN and its backward (the "expert" of the
// paper's Eq. (4) and its derivative in Eq. (5); Table 2 rows 11-13 name the
// tensors) is written as
//     C[m, n] = sum_kk A(m, kk) * B(n, kk)
// over one expert at a time, with the operands staged into LDS as 128-byte
// K-rows (64 bf16 or 32 fp32 values) and multiplied by 32x32 MFMA
// instructions (v_mfma_f32_32x32x16_bf16 / v_mfma_f32_32x32x2f32).
//
// Two kinds of operand loaders fill the LDS tiles:
//   RowLoader  operand rows whose K values are contiguous in HBM (activation
//              rows, weights used as W^T); optionally gathered through the
//              chunk's row->token table, so the dispatch never materialises
//              a permuted copy of X or dY.
//   ColLoader  operands whose K index is the slow HBM dimension (weights used
//              as W, and both operands of the weight gradients, whose K is
//              the expert's rows); each thread loads 4 K-rows x 16 bytes and
//              transposes them in registers before one LDS write per column.
// Tiles are 128 x 128 per 256-thread workgroup (2 x 2 waves of 64 x 64, i.e.
// 2 x 2 MFMA blocks per wave), K tiles are double-buffered in LDS with one
// barrier per K step, and LDS rows are XOR-swizzled in 16-byte units so the
// MFMA operand reads of 32 consecutive rows hit distinct banks.
//
// Scheduling on skewed expert loads: the row-grouped GEMMs (forward FC1/FC2,
// dgrads) enumerate m-tiles expert after expert from the chunk's offsets, so
// a cold expert costs only its own ceil(rows/128) tiles; the weight-gradient
// GEMMs (K = the expert's rows) visit experts in descending row count, the
// longest tiles first.
#include "common.h"
#include "kernels.h"

namespace memfine {
namespace {

constexpr int kBM = 128, kBN = 128, kThreads = 256;
constexpr int kRowBytes = 128;
constexpr int kTileBytes = (kBM + kBN) * kRowBytes;  // one A + one B stage: 32 KB

// byte offset of 16-byte unit `c` (0..7) of LDS tile row `row`
__device__ __forceinline__ int lds_off(int row, int c) {
  return row * kRowBytes + ((c ^ ((row ^ (row >> 3)) & 7)) << 4);
}

template <typename T> struct Mfma;
template <> struct Mfma<bf16_t> {
  static constexpr int kBK = 64;
  static constexpr int kKStep = 16;
  typedef bf16x8_t Frag;
  __device__ __forceinline__ static Frag read(const char* lds, int row, int kk, int lane) {
    const int c = kk * 2 + (lane >> 5);  // 8 K values = one 16-byte unit
    return *(const bf16x8_t*)(lds + lds_off(row, c));
  }
  __device__ __forceinline__ static void mma(const Frag& a, const Frag& b, f32x16_t& c) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mfma<float> {
  static constexpr int kBK = 32;
  static constexpr int kKStep = 2;
  typedef float Frag;
  __device__ __forceinline__ static Frag read(const char* lds, int row, int kk, int lane) {
    const int kel = kk * 2 + (lane >> 5);
    return *(const float*)(lds + lds_off(row, kel >> 2) + ((kel & 3) << 2));
  }
  __device__ __forceinline__ static void mma(const Frag& a, const Frag& b, f32x16_t& c) {
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

struct Tile {
  int e;      // expert
  int m0;     // first output row (row-grouped: chunk row; wgrad: weight row)
  int mrows;  // valid output rows in this tile
  int n0;     // first output column
  int K;      // reduction length
  int r0;     // wgrad: first chunk row of the expert
};

// ---------------------------------------------------------------- loaders
// 128 tile rows x 128 bytes; thread q-th unit: idx = tid + 256 q,
// row = idx >> 3, unit = idx & 7 (8 threads read one row's 128 bytes).
struct RowLoader {
  const char* ptr[4];
  u32x4_t reg[4];
  __device__ __forceinline__ void set_row(int q, const char* p) { ptr[q] = p; }
  __device__ __forceinline__ void fetch(int kt) {
    const int c = threadIdx.x & 7;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (ptr[q]) reg[q] = *(const u32x4_t*)(ptr[q] + (int64_t)kt * kRowBytes + c * 16);
      else reg[q] = u32x4_t{0u, 0u, 0u, 0u};
    }
  }
  __device__ __forceinline__ void store(char* lds) const {
    const int c = threadIdx.x & 7;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int row = (threadIdx.x + 256 * q) >> 3;
      *(u32x4_t*)(lds + lds_off(row, c)) = reg[q];
    }
  }
  __device__ __forceinline__ static int row_of(int q) { return (threadIdx.x + 256 * q) >> 3; }
};

// Operand with K as the slow dimension.  Thread (ng, kg): ng = tid % NG picks
// 16 bytes (V elements = V tile rows) of every K row, kg = tid / NG picks K
// rows 4kg .. 4kg+3 of the K tile.
template <typename T> struct ColLoader {
  static constexpr int V = Elem<T>::kVec;
  static constexpr int NG = 128 / V;
  u32x4_t reg[4];
  __device__ __forceinline__ static int ng() { return threadIdx.x % NG; }
  __device__ __forceinline__ static int kg() { return threadIdx.x / NG; }
  __device__ __forceinline__ void fetch(const char* const (&p)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (p[i]) reg[i] = *(const u32x4_t*)p[i];
      else reg[i] = u32x4_t{0u, 0u, 0u, 0u};
    }
  }
  __device__ __forceinline__ void store(char* lds) const;
};

template <> __device__ __forceinline__ void ColLoader<bf16_t>::store(char* lds) const {
  // 4 K values x 8 columns of bf16 -> per column 8 bytes (4 K values)
  const int n = ng(), g = kg();
  const int c = g >> 1, half = (g & 1) * 8;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t lo0 = (reg[0][j] & 0xffffu) | (reg[1][j] << 16);
    const uint32_t lo1 = (reg[2][j] & 0xffffu) | (reg[3][j] << 16);
    const uint32_t hi0 = (reg[0][j] >> 16) | (reg[1][j] & 0xffff0000u);
    const uint32_t hi1 = (reg[2][j] >> 16) | (reg[3][j] & 0xffff0000u);
    const int r0 = n * 8 + 2 * j, r1 = r0 + 1;
    *(u32x2_t*)(lds + lds_off(r0, c) + half) = u32x2_t{lo0, lo1};
    *(u32x2_t*)(lds + lds_off(r1, c) + half) = u32x2_t{hi0, hi1};
  }
}
template <> __device__ __forceinline__ void ColLoader<float>::store(char* lds) const {
  // 4 K values x 4 columns of fp32 -> per column one 16-byte unit
  const int n = ng(), g = kg();
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = n * 4 + j;
    *(u32x4_t*)(lds + lds_off(r, g)) = u32x4_t{reg[0][j], reg[1][j], reg[2][j], reg[3][j]};
  }
}

// --------------------------------------------------------------- compute
template <typename T>
__device__ __forceinline__ void mma_tile(const char* As, const char* Bs, f32x16_t (&acc)[2][2],
                                         int wm, int wn, int lane) {
  constexpr int KS = Mfma<T>::kBK / Mfma<T>::kKStep;
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    typename Mfma<T>::Frag a[2], b[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      a[i] = Mfma<T>::read(As, wm * 64 + i * 32 + (lane & 31), kk, lane);
      b[i] = Mfma<T>::read(Bs, wn * 64 + i * 32 + (lane & 31), kk, lane);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) Mfma<T>::mma(a[i], b[j], acc[i][j]);
  }
}

// Row (within the 128-row tile) of accumulator element i of MFMA block mb.
__device__ __forceinline__ int acc_row(int wm, int mb, int i, int lane) {
  return wm * 64 + mb * 32 + (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3);
}
__device__ __forceinline__ int acc_col(int wn, int nb, int lane) {
  return wn * 64 + nb * 32 + (lane & 31);
}

// m-tile bound for the row-grouped grid: sum_e ceil(c_e / 128) <= this.
inline int row_tiles_bound(int n, int E) { return (int)(((int64_t)n + (int64_t)E * (kBM - 1)) / kBM); }

// Expert and rows of m-tile `mt` of a row-grouped problem.
__device__ __forceinline__ bool locate_rows(const int32_t* __restrict__ offsets, int E, int mt,
                                            Tile& t) {
  int acc = 0;
  for (int e = 0; e < E; ++e) {
    const int r0 = offsets[e], r1 = offsets[e + 1];
    const int tiles = (r1 - r0 + kBM - 1) / kBM;
    if (mt < acc + tiles) {
      t.e = e;
      t.m0 = r0 + (mt - acc) * kBM;
      t.mrows = min(kBM, r1 - t.m0);
      return true;
    }
    acc += tiles;
  }
  return false;
}

template <typename T> __device__ __forceinline__ const char* cptr(const void* base, int64_t el) {
  return (const char*)base + el * (int64_t)sizeof(T);
}

// ================================================================ problems
// Forward FC1 + SwiGLU (and the backward's recompute of it).
//   A(m, kk) = X[tok(m0 + m), kk]            K = h  (gathered rows)
//   B(nr, kk) = W1[e, wrow(nr), kk]          tile column nr: waves own 64
//   columns each = 32 gate rows f and the 32 up rows F + f for the same f, so
//   every lane holds both halves of its SwiGLU pair.
template <typename T, bool kRecompute> struct ProbFC1 {
  RowLoader A, B;
  static int tiles_n(const GemmArgs& g) { return g.F / 64; }
  __device__ bool locate(const GemmArgs& g, Tile& t) const {
    const int ntn = g.F / 64;
    const int mt = blockIdx.x / ntn, nt = blockIdx.x % ntn;
    if (!locate_rows(g.offsets, g.E, mt, t)) return false;
    t.n0 = nt * 64;  // first f of the tile
    t.K = g.h;
    return true;
  }
  __device__ void init(const GemmArgs& g, const Tile& t) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = RowLoader::row_of(q);
      A.set_row(q, r < t.mrows ? cptr<T>(g.X, (int64_t)g.tok_of_row[t.m0 + r] * g.h) : nullptr);
      const int f = t.n0 + (r >> 6) * 32 + (r & 31);
      const int wrow = (r & 32) ? g.F + f : f;
      B.set_row(q, cptr<T>(g.W1, ((int64_t)t.e * 2 * g.F + wrow) * g.h));
    }
  }
  __device__ void fetch(const GemmArgs&, const Tile&, int kt) { A.fetch(kt); B.fetch(kt); }
  __device__ void store(char* As, char* Bs) const { A.store(As); B.store(Bs); }
  __device__ void epilogue(const GemmArgs& g, const Tile& t, const f32x16_t (&acc)[2][2], int wm,
                           int wn, int lane) const {
    const int f = t.n0 + wn * 32 + (lane & 31);
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int r = acc_row(wm, mb, i, lane);
        if (r >= t.mrows) continue;
        const int64_t row = t.m0 + r;
        const float gate = acc[mb][0][i], up = acc[mb][1][i];
        const float act = gate * sigmoidf_(gate) * up;
        if (!kRecompute) {
          Elem<T>::store((T*)g.a + row * g.F + f, act);
        } else {
          T* u = (T*)g.u + row * 2 * g.F;
          Elem<T>::store(u + f, gate);
          Elem<T>::store(u + g.F + f, up);
          Elem<T>::store((T*)g.ag + row * g.F + f, g.gate_of_row[row] * act);
        }
      }
  }
};

// Forward FC2: y[m, n] = sum_f a[m, f] W2[e, n, f].     K = F
template <typename T> struct ProbFC2 {
  RowLoader A, B;
  static int tiles_n(const GemmArgs& g) { return (g.h + kBN - 1) / kBN; }
  __device__ bool locate(const GemmArgs& g, Tile& t) const {
    const int ntn = (g.h + kBN - 1) / kBN;
    const int mt = blockIdx.x / ntn, nt = blockIdx.x % ntn;
    if (!locate_rows(g.offsets, g.E, mt, t)) return false;
    t.n0 = nt * kBN;
    t.K = g.F;
    return true;
  }
  __device__ void init(const GemmArgs& g, const Tile& t) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = RowLoader::row_of(q);
      A.set_row(q, r < t.mrows ? cptr<T>(g.a, (int64_t)(t.m0 + r) * g.F) : nullptr);
      const int n = t.n0 + r;
      B.set_row(q, n < g.h ? cptr<T>(g.W2, ((int64_t)t.e * g.h + n) * g.F) : nullptr);
    }
  }
  __device__ void fetch(const GemmArgs&, const Tile&, int kt) { A.fetch(kt); B.fetch(kt); }
  __device__ void store(char* As, char* Bs) const { A.store(As); B.store(Bs); }
  __device__ void epilogue(const GemmArgs& g, const Tile& t, const f32x16_t (&acc)[2][2], int wm,
                           int wn, int lane) const {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int n = t.n0 + acc_col(wn, nb, lane);
      if (n >= g.h) continue;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = acc_row(wm, mb, i, lane);
          if (r < t.mrows) Elem<T>::store((T*)g.y + (int64_t)(t.m0 + r) * g.h + n, acc[mb][nb][i]);
        }
    }
  }
};

// Backward FC2 dgrad with the SwiGLU backward and the gate-gradient partial
// fused into the epilogue:
//   dA[m, f] = sum_o dY[tok(m), o] W2[e, o, f]          K = h
//   a = silu(u_g) u_u;  da = g dA;  du_g = da u_u silu'(u_g);  du_u = da silu(u_g)
//   dgp[m, p] = sum over this wave's 64 columns of dA * a
// du overwrites u in place (each element is read and written by one lane).
template <typename T> struct ProbFC2Dgrad {
  RowLoader A;
  ColLoader<T> B;
  const char* bbase;  // W2[e] + this thread's column group
  bool bvalid;
  static int tiles_n(const GemmArgs& g) { return (g.F + kBN - 1) / kBN; }
  __device__ bool locate(const GemmArgs& g, Tile& t) const {
    const int ntn = (g.F + kBN - 1) / kBN;
    const int mt = blockIdx.x / ntn, nt = blockIdx.x % ntn;
    if (!locate_rows(g.offsets, g.E, mt, t)) return false;
    t.n0 = nt * kBN;
    t.K = g.h;
    return true;
  }
  __device__ void init(const GemmArgs& g, const Tile& t) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = RowLoader::row_of(q);
      A.set_row(q, r < t.mrows ? cptr<T>(g.dY, (int64_t)g.tok_of_row[t.m0 + r] * g.h) : nullptr);
    }
    const int n = t.n0 + ColLoader<T>::ng() * ColLoader<T>::V;
    bvalid = n < g.F;
    bbase = cptr<T>(g.W2, (int64_t)t.e * g.h * g.F + n);
  }
  __device__ void fetch(const GemmArgs& g, const Tile&, int kt) {
    A.fetch(kt);
    const char* p[4];
    const int k0 = kt * Mfma<T>::kBK + ColLoader<T>::kg() * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = bvalid ? bbase + (int64_t)(k0 + i) * g.F * sizeof(T) : nullptr;
    B.fetch(p);
  }
  __device__ void store(char* As, char* Bs) const { A.store(As); B.store(Bs); }
  __device__ void epilogue(const GemmArgs& g, const Tile& t, const f32x16_t (&acc)[2][2], int wm,
                           int wn, int lane) const {
    float part[2][16];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int i = 0; i < 16; ++i) part[mb][i] = 0.f;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int f = t.n0 + acc_col(wn, nb, lane);
      if (f >= g.F) continue;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = acc_row(wm, mb, i, lane);
          if (r >= t.mrows) continue;
          const int64_t row = t.m0 + r;
          T* u = (T*)g.u + row * 2 * g.F;
          const float ug = Elem<T>::load(u + f), uu = Elem<T>::load(u + g.F + f);
          const float s = sigmoidf_(ug), silu = ug * s;
          const float dA = acc[mb][nb][i];
          part[mb][i] = fmaf(dA, silu * uu, part[mb][i]);
          const float da = g.gate_of_row[row] * dA;
          Elem<T>::store(u + f, da * uu * s * (1.f + ug * (1.f - s)));
          Elem<T>::store(u + g.F + f, da * silu);
        }
    }
    // sum the partials over the 32 columns held by lanes with equal lane>>5
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float v = part[mb][i];
#pragma unroll
        for (int o = 1; o < 32; o <<= 1) v += __shfl_xor(v, o, 64);
        const int r = acc_row(wm, mb, i, lane);
        if ((lane & 31) == 0 && r < t.mrows)
          g.dgp[(int64_t)(t.m0 + r) * g.P + t.n0 / 64 + wn] = v;
      }
  }
};

// Backward FC1 dgrad: dxp[m, n] = sum_c du[m, c] W1[e, c, n].    K = 2F
template <typename T> struct ProbFC1Dgrad {
  RowLoader A;
  ColLoader<T> B;
  const char* bbase;
  bool bvalid;
  static int tiles_n(const GemmArgs& g) { return (g.h + kBN - 1) / kBN; }
  __device__ bool locate(const GemmArgs& g, Tile& t) const {
    const int ntn = (g.h + kBN - 1) / kBN;
    const int mt = blockIdx.x / ntn, nt = blockIdx.x % ntn;
    if (!locate_rows(g.offsets, g.E, mt, t)) return false;
    t.n0 = nt * kBN;
    t.K = 2 * g.F;
    return true;
  }
  __device__ void init(const GemmArgs& g, const Tile& t) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = RowLoader::row_of(q);
      A.set_row(q, r < t.mrows ? cptr<T>(g.u, (int64_t)(t.m0 + r) * 2 * g.F) : nullptr);
    }
    const int n = t.n0 + ColLoader<T>::ng() * ColLoader<T>::V;
    bvalid = n < g.h;
    bbase = cptr<T>(g.W1, (int64_t)t.e * 2 * g.F * g.h + n);
  }
  __device__ void fetch(const GemmArgs& g, const Tile&, int kt) {
    A.fetch(kt);
    const char* p[4];
    const int k0 = kt * Mfma<T>::kBK + ColLoader<T>::kg() * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) p[i] = bvalid ? bbase + (int64_t)(k0 + i) * g.h * sizeof(T) : nullptr;
    B.fetch(p);
  }
  __device__ void store(char* As, char* Bs) const { A.store(As); B.store(Bs); }
  __device__ void epilogue(const GemmArgs& g, const Tile& t, const f32x16_t (&acc)[2][2], int wm,
                           int wn, int lane) const {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int n = t.n0 + acc_col(wn, nb, lane);
      if (n >= g.h) continue;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = acc_row(wm, mb, i, lane);
          if (r < t.mrows) Elem<T>::store((T*)g.dxp + (int64_t)(t.m0 + r) * g.h + n, acc[mb][nb][i]);
        }
    }
  }
};

// Weight gradients.  Expert e's rows [r0, r0 + K) are the reduction axis:
//   FC2: dW2[e, m, n] (+)= sum_r dY[tok(r), m] * ag[r, n]     M = h,  N = F
//   FC1: dW1[e, m, n] (+)= sum_r du[r, m] * X[tok(r), n]      M = 2F, N = h
// Both operands are ColLoaders; tile (rank, mt, nt) with experts visited in
// descending row count.
template <typename T, bool kFC1> struct ProbWgrad {
  ColLoader<T> A, B;
  const char* abase;
  const char* bbase;
  bool avalid, bvalid;
  __host__ __device__ static int M(const GemmArgs& g) { return kFC1 ? 2 * g.F : g.h; }
  __host__ __device__ static int N(const GemmArgs& g) { return kFC1 ? g.h : g.F; }
  static int tiles(const GemmArgs& g) {
    return g.E * ((M(g) + kBM - 1) / kBM) * ((N(g) + kBN - 1) / kBN);
  }
  __device__ bool locate(const GemmArgs& g, Tile& t) const {
    const int mtn = (M(g) + kBM - 1) / kBM, ntn = (N(g) + kBN - 1) / kBN;
    const int per = mtn * ntn;
    const int rank = blockIdx.x / per, rem = blockIdx.x % per;
    t.e = g.order[rank];
    t.r0 = g.offsets[t.e];
    t.K = g.offsets[t.e + 1] - t.r0;
    if (t.K == 0 && g.accumulate) return false;  // nothing to add
    t.m0 = (rem / ntn) * kBM;
    t.n0 = (rem % ntn) * kBN;
    t.mrows = min(kBM, M(g) - t.m0);
    return true;
  }
  __device__ void init(const GemmArgs& g, const Tile& t) {
    const int ma = t.m0 + ColLoader<T>::ng() * ColLoader<T>::V;
    const int nb = t.n0 + ColLoader<T>::ng() * ColLoader<T>::V;
    avalid = ma < M(g);
    bvalid = nb < N(g);
    abase = kFC1 ? cptr<T>(g.u, ma) : cptr<T>(g.dY, ma);
    bbase = kFC1 ? cptr<T>(g.X, nb) : cptr<T>(g.ag, nb);
  }
  __device__ void fetch(const GemmArgs& g, const Tile& t, int kt) {
    const char* pa[4];
    const char* pb[4];
    const int k0 = kt * Mfma<T>::kBK + ColLoader<T>::kg() * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int kk = k0 + i;
      const bool in = kk < t.K;
      const int row = t.r0 + (in ? kk : 0);
      if (kFC1) {
        pa[i] = (in && avalid) ? abase + (int64_t)row * 2 * g.F * sizeof(T) : nullptr;
        pb[i] = (in && bvalid) ? bbase + (int64_t)g.tok_of_row[row] * g.h * sizeof(T) : nullptr;
      } else {
        pa[i] = (in && avalid) ? abase + (int64_t)g.tok_of_row[row] * g.h * sizeof(T) : nullptr;
        pb[i] = (in && bvalid) ? bbase + (int64_t)row * g.F * sizeof(T) : nullptr;
      }
    }
    A.fetch(pa);
    B.fetch(pb);
  }
  __device__ void store(char* As, char* Bs) const { A.store(As); B.store(Bs); }
  __device__ void epilogue(const GemmArgs& g, const Tile& t, const f32x16_t (&acc)[2][2], int wm,
                           int wn, int lane) const {
    float* dW = (kFC1 ? g.dW1 : g.dW2) + (int64_t)t.e * M(g) * N(g);
    const int Nn = N(g);
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const int n = t.n0 + acc_col(wn, nb, lane);
      if (n >= Nn) continue;
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = acc_row(wm, mb, i, lane);
          if (r >= t.mrows) continue;
          float* p = dW + (int64_t)(t.m0 + r) * Nn + n;
          *p = g.accumulate ? *p + acc[mb][nb][i] : acc[mb][nb][i];
        }
    }
  }
};

// ------------------------------------------------------------------ kernel
template <typename T, class P>
__global__ __launch_bounds__(kThreads, 2) void grouped_gemm_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) char smem[2 * kTileBytes];
  P p;
  Tile t;
  if (!p.locate(g, t)) return;
  p.init(g, t);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wm = w >> 1, wn = w & 1;
  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;
  const int nk = (t.K + Mfma<T>::kBK - 1) / Mfma<T>::kBK;
  if (nk > 0) {
    p.fetch(g, t, 0);
    p.store(smem, smem + kBM * kRowBytes);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      char* cur = smem + (kt & 1) * kTileBytes;
      char* nxt = smem + ((kt + 1) & 1) * kTileBytes;
      if (kt + 1 < nk) p.fetch(g, t, kt + 1);
      mma_tile<T>(cur, cur + kBM * kRowBytes, acc, wm, wn, lane);
      if (kt + 1 < nk) p.store(nxt, nxt + kBM * kRowBytes);
      __syncthreads();
    }
  }
  p.epilogue(g, t, acc, wm, wn, lane);
}

template <class PB, class PF>
hipError_t launch_grid(const GemmArgs& g, int blocks, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  if (g.dtype == 0) grouped_gemm_kernel<bf16_t, PB><<<blocks, kThreads, 0, s>>>(g);
  else grouped_gemm_kernel<float, PF><<<blocks, kThreads, 0, s>>>(g);
  return hipGetLastError();
}

}  // namespace

int dgate_partials(int F) { return 2 * ((F + kBN - 1) / kBN); }

hipError_t launch_fc1_fwd(const GemmArgs& g, hipStream_t s) {
  return launch_grid<ProbFC1<bf16_t, false>, ProbFC1<float, false>>(
      g, row_tiles_bound(g.n, g.E) * (g.F / 64), s);
}
hipError_t launch_fc1_recompute(const GemmArgs& g, hipStream_t s) {
  return launch_grid<ProbFC1<bf16_t, true>, ProbFC1<float, true>>(
      g, row_tiles_bound(g.n, g.E) * (g.F / 64), s);
}
hipError_t launch_fc2_fwd(const GemmArgs& g, hipStream_t s) {
  return launch_grid<ProbFC2<bf16_t>, ProbFC2<float>>(
      g, row_tiles_bound(g.n, g.E) * ((g.h + kBN - 1) / kBN), s);
}
hipError_t launch_fc2_dgrad(const GemmArgs& g, hipStream_t s) {
  return launch_grid<ProbFC2Dgrad<bf16_t>, ProbFC2Dgrad<float>>(
      g, row_tiles_bound(g.n, g.E) * ((g.F + kBN - 1) / kBN), s);
}
hipError_t launch_fc1_dgrad(const GemmArgs& g, hipStream_t s) {
  return launch_grid<ProbFC1Dgrad<bf16_t>, ProbFC1Dgrad<float>>(
      g, row_tiles_bound(g.n, g.E) * ((g.h + kBN - 1) / kBN), s);
}
hipError_t launch_fc2_wgrad(const GemmArgs& g, hipStream_t s) {
  return launch_grid<ProbWgrad<bf16_t, false>, ProbWgrad<float, false>>(
      g, ProbWgrad<float, false>::tiles(g), s);
}
hipError_t launch_fc1_wgrad(const GemmArgs& g, hipStream_t s) {
  return launch_grid<ProbWgrad<bf16_t, true>, ProbWgrad<float, true>>(
      g, ProbWgrad<float, true>::tiles(g), s);
}

}  // namespace memfine
