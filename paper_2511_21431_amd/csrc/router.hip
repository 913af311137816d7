// Router in front of the expert layer on gfx950: logits = X Wr^T on the
// matrix cores, softmax, top-k and renormalised gates in registers; the
// backward's per-token gate-to-logit gradient, its dX contribution, and the
// reduction of partial weight gradients.  (Table 2 rows 9-10 store the
// router's input and its logits; the gates are the scores that multiply the
// expert outputs.)
#include "common.h"
#include "kernels.h"

namespace memfine {
namespace {

constexpr int kRouterWaves = 4;   // one 32-token block per workgroup, K split over the waves

// Per-lane K layout of one K block.  Lane l (row l % 32, half l / 32) holds a
// contiguous half of its row's block: for bf16 the block is 64 elements and
// the lane holds elements [32 (l/32), 32 (l/32) + 32) as four 16-byte
// fragments, fragment s feeding MFMA step s (K 16 split as 8 + 8 over the two
// lane halves).  A and B use the same map, so each step sums a disjoint part
// of the block.  For fp32 the block is 32 elements, the lane holds 16 of them
// and step s takes its s-th element (K 2 split as 1 + 1).
template <typename T> struct RK;
template <> struct RK<bf16_t> {
  static constexpr int KB = 64, STEPS = 4;
  typedef u32x4_t Raw[4];
  __device__ __forceinline__ static void load(const bf16_t* row, int kb, int hh, Raw& r) {
    const u32x4_t* p = (const u32x4_t*)(row + kb * KB + 32 * hh);
#pragma unroll
    for (int s = 0; s < 4; ++s) r[s] = p[s];
  }
  __device__ __forceinline__ static void mma(const Raw& a, const Raw& b, f32x16_t& c) {
#pragma unroll
    for (int s = 0; s < 4; ++s)
      c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, b[s]),
                                                  __builtin_bit_cast(bf16x8_t, a[s]), c, 0, 0, 0);
  }
};
template <> struct RK<float> {
  static constexpr int KB = 32, STEPS = 16;
  typedef f32x4_t Raw[4];
  __device__ __forceinline__ static void load(const float* row, int kb, int hh, Raw& r) {
    const f32x4_t* p = (const f32x4_t*)(row + kb * KB + 16 * hh);
#pragma unroll
    for (int s = 0; s < 4; ++s) r[s] = p[s];
  }
  __device__ __forceinline__ static void mma(const Raw& a, const Raw& b, f32x16_t& c) {
#pragma unroll
    for (int s = 0; s < 16; ++s)
      c = __builtin_amdgcn_mfma_f32_32x32x2f32(b[s >> 2][s & 3], a[s >> 2][s & 3], c, 0, 0, 0);
  }
};

// Forward.  A workgroup owns 32 tokens x 32 NB experts (NB = 1 or 2); its
// four waves take interleaved K blocks (wave w: blocks w, w + 4, ...) with the
// operands loaded straight into registers one block ahead, and wave 0 sums
// the four partial products through LDS.  After that lane l of wave 0 holds, for token l % 32, the logits of experts
// 32 nb + 8 (q / 4) + 4 (l / 32) + q % 4 (q = 0..15); lane l ^ 32 holds the
// token's other half.  Top-k: k rounds, each lane proposes its largest
// unselected logit (equal: lower id), the two halves compare over one
// shuffle, the owner marks the winner.
template <typename T, int NB>
__global__ __launch_bounds__(64 * kRouterWaves) void router_fwd_kernel(
    const T* __restrict__ X, const T* __restrict__ Wr, int64_t T_, int h, int E, int k,
    int32_t* __restrict__ idx, float* __restrict__ gates, float* __restrict__ logits) {
  typedef RK<T> K;
  __shared__ f32x16_t part[kRouterWaves - 1][NB][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r = lane & 31, hh = lane >> 5;
  const int64_t t0 = (int64_t)blockIdx.x * 32;
  const int64_t trow = min(t0 + r, T_ - 1);  // rows past T read the last row
  const T* xr = X + trow * h;
  const T* wr[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) wr[nb] = Wr + (int64_t)min(32 * nb + r, E - 1) * h;
  f32x16_t acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[nb][q] = 0.f;
  typename K::Raw a[2], b[2][NB];
  const int nkb = h / K::KB;
  constexpr int W = kRouterWaves;
  // this wave's K blocks: w, w + W, w + 2W, ...
  if (w < nkb) {
    K::load(xr, w, hh, a[0]);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) K::load(wr[nb], w, hh, b[0][nb]);
  }
  for (int kb = w; kb < nkb; kb += 2 * W) {
    if (kb + W < nkb) {
      K::load(xr, kb + W, hh, a[1]);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) K::load(wr[nb], kb + W, hh, b[1][nb]);
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) K::mma(a[0], b[0][nb], acc[nb]);
    if (kb + W >= nkb) break;
    if (kb + 2 * W < nkb) {
      K::load(xr, kb + 2 * W, hh, a[0]);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) K::load(wr[nb], kb + 2 * W, hh, b[0][nb]);
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) K::mma(a[1], b[1][nb], acc[nb]);
  }
  // partial products of waves 1..W-1 to LDS, summed by wave 0 in wave order
  if (w > 0) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) part[w - 1][nb][lane] = acc[nb];
  }
  __syncthreads();
  if (w > 0) return;
#pragma unroll
  for (int ww = 0; ww < W - 1; ++ww)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] += part[ww][nb][lane];
  const bool live = t0 + r < T_;
  const int64_t t = t0 + r;
  // expert id of element q of block nb held by this lane
  auto col = [&](int nb, int q) { return 32 * nb + 8 * (q >> 2) + 4 * hh + (q & 3); };
  if (logits && live) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int q = 0; q < 16; ++q)
        if (col(nb, q) < E) logits[t * E + col(nb, q)] = acc[nb][q];
  }
  uint32_t taken[NB] = {};
  float selv[16];
  int seli[16];
  for (int j = 0; j < k; ++j) {
    float bv = -INFINITY;
    int bi = INT32_MAX;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int c = col(nb, q);
        const bool ok = c < E && !((taken[nb] >> q) & 1u);
        const float v = acc[nb][q];
        if (ok && (v > bv || (v == bv && c < bi))) {
          bv = v;
          bi = c;
        }
      }
    const float ov = __shfl_xor(bv, 32, 64);
    const int oi = __shfl_xor(bi, 32, 64);
    if (ov > bv || (ov == bv && oi < bi)) {
      bv = ov;
      bi = oi;
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int q = 0; q < 16; ++q)
        if (col(nb, q) == bi) taken[nb] |= 1u << q;
#pragma unroll
    for (int jj = 0; jj < 16; ++jj)
      if (jj == j) {
        selv[jj] = bv;
        seli[jj] = bi;
      }
  }
  if (hh == 0 && live) {
    // renormalised softmax over the selected logits (the full softmax's
    // denominator cancels); selv[0] is the largest
    float e[16], sum = 0.f;
#pragma unroll
    for (int jj = 0; jj < 16; ++jj) {
      e[jj] = jj < k ? __expf(selv[jj] - selv[0]) : 0.f;
      sum += e[jj];
    }
    const float inv = 1.f / sum;
#pragma unroll
    for (int jj = 0; jj < 16; ++jj)
      if (jj < k) {
        idx[t * k + jj] = seli[jj];
        gates[t * k + jj] = e[jj] * inv;
      }
  }
}

// Lane j's value, in a scalar register (uniform).
__device__ __forceinline__ float lane_value(float v, int j) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), j));
}
// One step of a (value, lower index) arg-max with the lane that DPP control
// `kCtrl` names (a permutation inside each row of 16 lanes).
template <int kCtrl>
__device__ __forceinline__ void argmax_dpp(float& v, int& i) {
  const float ov = __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), kCtrl, 0xf, 0xf, false));
  const int oi = __builtin_amdgcn_update_dpp(0, i, kCtrl, 0xf, 0xf, false);
  if (ov > v || (ov == v && oi < i)) {
    v = ov;
    i = oi;
  }
}
// The wave's arg-max over (value, lower index), left in every lane: inside
// each row of 16 lanes by DPP (swap neighbours, swap pairs, mirror halves of
// 8, mirror the row: after each step a lane holds the best of 2, 4, 8, 16
// lanes), then the four rows' results through scalar registers.
__device__ __forceinline__ void wave_argmax(float& v, int& i) {
  argmax_dpp<0xb1>(v, i);   // quad_perm [1, 0, 3, 2]
  argmax_dpp<0x4e>(v, i);   // quad_perm [2, 3, 0, 1]
  argmax_dpp<0x141>(v, i);  // row_half_mirror
  argmax_dpp<0x140>(v, i);  // row_mirror
  float bv = lane_value(v, 0);
  int bi = __builtin_amdgcn_readlane(i, 0);
#pragma unroll
  for (int r = 16; r < 64; r += 16) {
    const float ov = lane_value(v, r);
    const int oi = __builtin_amdgcn_readlane(i, r);
    if (ov > bv || (ov == bv && oi < bi)) {
      bv = ov;
      bi = oi;
    }
  }
  v = bv;
  i = bi;
}

// Top-k of one token whose logits a wave holds (lane l: experts l + 64 q,
// q < V; entries of experts >= E are ignored): k rounds of a wave-wide
// arg-max over (logit, lower id), so the selection and its order are those
// of the narrow kernel; then lanes 0..k-1 write the
// selected ids, largest first, and the gates renormalised over them (the
// full softmax's denominator cancels).
template <int V>
__device__ __forceinline__ void wave_topk(const float (&v)[V], int E, int k, int lane, int64_t t,
                                          int32_t* __restrict__ idx, float* __restrict__ gates) {
  uint32_t taken = 0;
  float selv[16];
  int seli[16];
  for (int j = 0; j < k; ++j) {
    float bv = -INFINITY;
    int bi = INT32_MAX;
#pragma unroll
    for (int q = 0; q < V; ++q) {
      const int e = lane + 64 * q;
      if (e < E && !((taken >> q) & 1u) && (v[q] > bv || (v[q] == bv && e < bi))) {
        bv = v[q];
        bi = e;
      }
    }
    wave_argmax(bv, bi);
    if ((bi & 63) == lane) taken |= 1u << (bi >> 6);
#pragma unroll
    for (int jj = 0; jj < 16; ++jj)
      if (jj == j) {
        selv[jj] = bv;
        seli[jj] = bi;
      }
  }
  // renormalised softmax over the selected logits; selv[0] is the largest
  float e[16], sum = 0.f;
#pragma unroll
  for (int jj = 0; jj < 16; ++jj) {
    e[jj] = jj < k ? __expf(selv[jj] - selv[0]) : 0.f;
    sum += e[jj];
  }
  const float inv = 1.f / sum;
#pragma unroll
  for (int jj = 0; jj < 16; ++jj)
    if (jj < k && lane == jj) {
      idx[t * k + jj] = seli[jj];
      gates[t * k + jj] = e[jj] * inv;
    }
}

// Forward for wide routers (64 < E <= 256 logits per token, the width of a
// 256-expert model).  A workgroup owns 32 tokens; wave w multiplies them
// with expert blocks w NBW .. w NBW + NBW - 1 (32 experts each) over the
// whole K, operands loaded straight into registers one K block ahead.  The
// logits go to LDS; then each wave selects the top-k of 8 of the tokens,
// one token at a time: lane l holds experts l, l + 64, l + 128, l + 192,
// and each of the k rounds is a wave-wide arg-max over (logit, lower id)
// by shuffles, so the selection and its order are those of the narrow
// kernel.
template <typename T, int NBW>
__global__ __launch_bounds__(64 * kRouterWaves) void router_fwd_wide_kernel(
    const T* __restrict__ X, const T* __restrict__ Wr, int64_t T_, int h, int E, int k,
    int32_t* __restrict__ idx, float* __restrict__ gates, float* __restrict__ logits) {
  typedef RK<T> K;
  constexpr int kMaxE = 32 * NBW * kRouterWaves;
  __shared__ float lg[32][kMaxE + 1];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r = lane & 31, hh = lane >> 5;
  const int64_t t0 = (int64_t)blockIdx.x * 32;
  const int64_t trow = min(t0 + r, T_ - 1);  // rows past T read the last row
  const T* xr = X + trow * h;
  const T* wr[NBW];
#pragma unroll
  for (int nb = 0; nb < NBW; ++nb)
    wr[nb] = Wr + (int64_t)min(32 * (w * NBW + nb) + r, E - 1) * h;
  f32x16_t acc[NBW];
#pragma unroll
  for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[nb][q] = 0.f;
  const bool any = 32 * w * NBW < E;  // a wave past the last expert block skips the product
  typename K::Raw a[2], b[2][NBW];
  const int nkb = h / K::KB;
  if (any) {
    K::load(xr, 0, hh, a[0]);
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) K::load(wr[nb], 0, hh, b[0][nb]);
    for (int kb = 0; kb < nkb; kb += 2) {
      if (kb + 1 < nkb) {
        K::load(xr, kb + 1, hh, a[1]);
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) K::load(wr[nb], kb + 1, hh, b[1][nb]);
      }
#pragma unroll
      for (int nb = 0; nb < NBW; ++nb) K::mma(a[0], b[0][nb], acc[nb]);
      if (kb + 1 >= nkb) break;
      if (kb + 2 < nkb) {
        K::load(xr, kb + 2, hh, a[0]);
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) K::load(wr[nb], kb + 2, hh, b[0][nb]);
      }
#pragma unroll
      for (int nb = 0; nb < NBW; ++nb) K::mma(a[1], b[1][nb], acc[nb]);
    }
  }
  // lane l holds, for token l % 32, experts 32 blk + 8 (q / 4) + 4 (l / 32) + q % 4
#pragma unroll
  for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
    for (int q = 0; q < 16; ++q)
      lg[r][32 * (w * NBW + nb) + 8 * (q >> 2) + 4 * hh + (q & 3)] = acc[nb][q];
  __syncthreads();
  constexpr int V = kMaxE / 64;  // logits per lane per token
  for (int tt = 0; tt < 32 / kRouterWaves; ++tt) {
    const int tok = w * (32 / kRouterWaves) + tt;
    const int64_t t = t0 + tok;
    if (t >= T_) break;  // uniform over the wave
    float v[V];
#pragma unroll
    for (int j = 0; j < V; ++j) {
      const int e = lane + 64 * j;
      v[j] = lg[tok][e];
      if (logits && e < E) logits[t * E + e] = v[j];
    }
    wave_topk<V>(v, E, k, lane, t, idx, gates);
  }
}

// Top-k of logits already in memory (fp32 [T, E], 64 < E <= 256), one wave
// per token, with the selection and gates of the kernels above: the router's
// second step when the logits come from the grouped GEMM.
__global__ __launch_bounds__(256) void router_topk_kernel(const float* __restrict__ logits,
                                                          int64_t T_, int E, int k,
                                                          int32_t* __restrict__ idx,
                                                          float* __restrict__ gates) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T_) return;  // uniform over the wave
  constexpr int V = 4;
  float v[V];
#pragma unroll
  for (int j = 0; j < V; ++j) {
    const int e = lane + 64 * j;
    v[j] = e < E ? logits[t * E + e] : 0.f;
  }
  wave_topk<V>(v, E, k, lane, t, idx, gates);
}

// Backward, one wave per token (grid-stride): dz_j = g_j (dg_j - sum g dg);
// dX[t] (+)= sum_j dz_j Wr[i_j]; the dense row D[t, 0..EP) = dz scattered to
// the selected experts (bf16 or fp32, zero elsewhere) for the weight-gradient
// GEMM.  Lane j < k loads slot j and the k values are broadcast by shuffles;
// each lane then covers NV vectors of the row per pass with their loads
// issued together.
template <typename T>
__global__ __launch_bounds__(256) void router_bwd_dx_kernel(
    const T* __restrict__ Wr, const int32_t* __restrict__ idx, const float* __restrict__ gates,
    const float* __restrict__ dgates, int64_t T_, int h, int E, int k, int EP, int accumulate,
    int with_dx, T* __restrict__ dX, T* __restrict__ D) {
  constexpr int V = Elem<T>::kVec;  // elements per 16-byte vector
  constexpr int NV = 4;             // vectors per lane per pass
  const int lane = threadIdx.x & 63;
  const int64_t waves = (int64_t)gridDim.x * 4;
  for (int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); t < T_; t += waves) {
    // slot `lane` (lanes < k); a slot whose id lies outside [0, E) is dropped
    const int i = lane < k ? idx[t * k + lane] : -1;
    const bool in = i >= 0 && i < E;
    const float g = in ? gates[t * k + lane] : 0.f, d = in ? dgates[t * k + lane] : 0.f;
    // sum over the k <= 16 slots held by lanes 0..15, read into scalar
    // registers (v_readlane) and added as a pairwise tree
    float gd[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) gd[j] = lane_value(g * d, j);
#pragma unroll
    for (int w = 1; w < 16; w <<= 1)
#pragma unroll
      for (int j = 0; j < 16; j += 2 * w) gd[j] += gd[j + w];
    const float c = gd[0];
    const float dz = g * (d - c);
    const int id = in ? i : -1;
    // the k slots, broadcast while every lane is active (the row loops below
    // leave lanes idle when h or EP is short)
    float dzs[16];
    int ids[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      dzs[j] = lane_value(dz, j);
      ids[j] = j < k ? __builtin_amdgcn_readlane(id, j) : -1;
    }
    for (int c0 = lane * V; with_dx && c0 < h; c0 += 64 * V * NV) {
      float acc[NV][V];
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int cc = c0 + v * 64 * V;
        if (accumulate && cc < h) {
          unpack16(*(const u32x4_t*)(dX + t * h + cc), acc[v], (T*)nullptr);
        } else {
#pragma unroll
          for (int q = 0; q < V; ++q) acc[v][q] = 0.f;
        }
      }
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float dzj = dzs[j];
        const int idj = ids[j];
        if (idj < 0) continue;
        u32x4_t wv[NV];
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          const int cc = c0 + v * 64 * V;
          wv[v] = *(const u32x4_t*)(Wr + (int64_t)idj * h + (cc < h ? cc : 0));
        }
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          float w[V];
          unpack16(wv[v], w, (T*)nullptr);
#pragma unroll
          for (int q = 0; q < V; ++q) acc[v][q] = fmaf(dzj, w[q], acc[v][q]);
        }
      }
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int cc = c0 + v * 64 * V;
        if (cc < h) *(u32x4_t*)(dX + t * h + cc) = pack16(acc[v], (T*)nullptr);
      }
    }
    for (int e0 = lane * V; e0 < EP; e0 += 64 * V) {
      float v[V];
#pragma unroll
      for (int q = 0; q < V; ++q) v[q] = 0.f;
#pragma unroll
      for (int j = 0; j < 16; ++j)
#pragma unroll
        for (int q = 0; q < V; ++q)
          if (ids[j] == e0 + q) v[q] += dzs[j];
      *(u32x4_t*)(D + t * EP + e0) = pack16(v, (T*)nullptr);
    }
  }
}

// dWr[e, n] (+)= sum over splits s of P[s, e, n], e < E (fixed order).
__global__ __launch_bounds__(256) void router_reduce_kernel(const float* __restrict__ P, int S,
                                                            int EP, int E, int h, int accumulate,
                                                            float* __restrict__ dWr) {
  const int64_t n4 = (int64_t)E * h / 4;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n4) return;
  const int64_t el = i * 4;
  const int e = (int)(el / h), n = (int)(el % h);
  f32x4_t acc = accumulate ? *(const f32x4_t*)(dWr + el) : (f32x4_t){0.f, 0.f, 0.f, 0.f};
  const float* p = P + (int64_t)e * h + n;
  const int64_t stride = (int64_t)EP * h;
  int s = 0;
  for (; s + 4 <= S; s += 4) {  // four loads in flight, summed in split order
    const f32x4_t v0 = *(const f32x4_t*)(p + (s + 0) * stride);
    const f32x4_t v1 = *(const f32x4_t*)(p + (s + 1) * stride);
    const f32x4_t v2 = *(const f32x4_t*)(p + (s + 2) * stride);
    const f32x4_t v3 = *(const f32x4_t*)(p + (s + 3) * stride);
    acc += v0;
    acc += v1;
    acc += v2;
    acc += v3;
  }
  for (; s < S; ++s) acc += *(const f32x4_t*)(p + s * stride);
  *(f32x4_t*)(dWr + el) = acc;
}

__global__ void iota_kernel(int32_t* p, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = i;
}
__global__ void split_offsets_kernel(int32_t* offsets, int32_t* order, int64_t T_, int S) {
  const int s = blockIdx.x * 256 + threadIdx.x;
  if (s <= S) offsets[s] = (int32_t)(s * T_ / S);
  if (s < S) order[s] = s;
}

}  // namespace

hipError_t launch_router_fwd(int dtype, const void* X, const void* Wr, int64_t T, int h, int E,
                             int k, int32_t* idx, float* gates, float* logits, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int blocks = (int)((T + 31) / 32);
  const dim3 grid(blocks), block(64 * kRouterWaves);
  if (dtype == 0) {
    const bf16_t *x = (const bf16_t*)X, *wr = (const bf16_t*)Wr;
    if (E <= 32)
      router_fwd_kernel<bf16_t, 1><<<grid, block, 0, s>>>(x, wr, T, h, E, k, idx, gates, logits);
    else if (E <= 64)
      router_fwd_kernel<bf16_t, 2><<<grid, block, 0, s>>>(x, wr, T, h, E, k, idx, gates, logits);
    else if (E <= 128)
      router_fwd_wide_kernel<bf16_t, 1><<<grid, block, 0, s>>>(x, wr, T, h, E, k, idx, gates, logits);
    else
      router_fwd_wide_kernel<bf16_t, 2><<<grid, block, 0, s>>>(x, wr, T, h, E, k, idx, gates, logits);
  } else {
    const float *x = (const float*)X, *wr = (const float*)Wr;
    if (E <= 32)
      router_fwd_kernel<float, 1><<<grid, block, 0, s>>>(x, wr, T, h, E, k, idx, gates, logits);
    else if (E <= 64)
      router_fwd_kernel<float, 2><<<grid, block, 0, s>>>(x, wr, T, h, E, k, idx, gates, logits);
    else if (E <= 128)
      router_fwd_wide_kernel<float, 1><<<grid, block, 0, s>>>(x, wr, T, h, E, k, idx, gates, logits);
    else
      router_fwd_wide_kernel<float, 2><<<grid, block, 0, s>>>(x, wr, T, h, E, k, idx, gates, logits);
  }
  return hipGetLastError();
}

hipError_t launch_router_topk(const float* logits, int64_t T, int E, int k, int32_t* idx,
                              float* gates, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (E > 256 || k > 16) return hipErrorInvalidValue;
  router_topk_kernel<<<(unsigned)((T + 3) / 4), 256, 0, s>>>(logits, T, E, k, idx, gates);
  return hipGetLastError();
}

hipError_t launch_router_bwd_dx(int dtype, const void* Wr, const int32_t* idx, const float* gates,
                                const float* dgates, int64_t T, int h, int E, int k, int EP,
                                int accumulate, int with_dx, void* dX, void* D, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int64_t want = (T + 3) / 4;
  const int blocks = (int)(want < 8192 ? want : 8192);
  if (dtype == 0)
    router_bwd_dx_kernel<bf16_t><<<blocks, 256, 0, s>>>((const bf16_t*)Wr, idx, gates, dgates, T, h, E, k, EP, accumulate, with_dx, (bf16_t*)dX, (bf16_t*)D);
  else
    router_bwd_dx_kernel<float><<<blocks, 256, 0, s>>>((const float*)Wr, idx, gates, dgates, T, h, E, k, EP, accumulate, with_dx, (float*)dX, (float*)D);
  return hipGetLastError();
}

hipError_t launch_router_split_meta(int32_t* offsets, int32_t* order, int32_t* tok, int64_t T, int S,
                                    hipStream_t s) {
  split_offsets_kernel<<<(S + 1 + 255) / 256, 256, 0, s>>>(offsets, order, T, S);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || T == 0) return e;
  iota_kernel<<<(int)((T + 255) / 256), 256, 0, s>>>(tok, (int)T);
  return hipGetLastError();
}

hipError_t launch_router_reduce(const float* P, int S, int EP, int E, int h, int accumulate,
                                float* dWr, hipStream_t s) {
  const int64_t n4 = (int64_t)E * h / 4;
  if (n4 == 0) return hipSuccess;
  router_reduce_kernel<<<(int)((n4 + 255) / 256), 256, 0, s>>>(P, S, EP, E, h, accumulate, dWr);
  return hipGetLastError();
}

}  // namespace memfine
