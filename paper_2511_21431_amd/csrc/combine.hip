// Memory-bound gather/sum kernels of the chunked MoE layer.
//
// combine:    the gate-weighted sum over a token's k slots that follows the
//             expert (Table 2 "score mul" and "add"; the "combine" of
//             Eq. (4)): Y[t] = sum_j g[t,j] * y[row(t,j)], j ascending, fp32.
// unpermute:  its backward for the input gradient, dX[t] = sum_j dxp[row(t,j)]
//             (the concatenation of Eq. (7) fills dX chunk by chunk), and the
//             gate gradient dg[t,j] = sum of the per-tile partial dot products
//             the FC2 backward kernel leaves for row(t,j).
// Each thread moves one 16-byte vector of a row; consecutive threads take
// consecutive vectors, so every row is read and written with full coalescing.
// A token's slots are taken 8 at a time: their row ids first, then all their
// vector loads, so the loads of one group are in flight together.
#include "common.h"
#include "kernels.h"

namespace memfine {

template <typename T>
__global__ __launch_bounds__(256) void combine_kernel(const T* __restrict__ y,
                                                      const int32_t* __restrict__ row_of_slot,
                                                      const float* __restrict__ gates, int64_t t0,
                                                      int tokens, int h, int k,
                                                      T* __restrict__ Y) {
  constexpr int V = Elem<T>::kVec;
  const int vpr = h / V;
  const int64_t gid = blockIdx.x * 256ll + threadIdx.x;
  if (gid >= (int64_t)tokens * vpr) return;
  const int i = (int)(gid / vpr), c = (int)(gid % vpr);
  const int64_t t = t0 + i;
  float acc[V];
#pragma unroll
  for (int q = 0; q < V; ++q) acc[q] = 0.f;
  for (int j0 = 0; j0 < k; j0 += 8) {
    int r[8];
    float g[8];
    u32x4_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const bool in = j0 + j < k;
      r[j] = in ? row_of_slot[(int64_t)i * k + j0 + j] : -1;
      g[j] = in ? gates[t * k + j0 + j] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)  // (k is uniform: no load past the token's slots;
      if (j0 + j < k)            // a dropped slot, r < 0, reads row 0 with weight 0)
        v[j] = *(const u32x4_t*)(y + (int64_t)(r[j] < 0 ? 0 : r[j]) * h + c * V);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (r[j] < 0) continue;
      float f[V];
      unpack16(v[j], f, (T*)nullptr);
#pragma unroll
      for (int q = 0; q < V; ++q) acc[q] = fmaf(g[j], f[q], acc[q]);
    }
  }
  *(u32x4_t*)(Y + t * h + c * V) = pack16(acc, (T*)nullptr);
}

// sum of the P per-tile partials of one row, in index order (P = F / 32 is
// even: 8-byte loads); 0 for a dropped slot (r < 0)
__device__ __forceinline__ float dgate_of_row(const float* __restrict__ dgp, int P, int r) {
  float s = 0.f;
  if (r >= 0) {
    const f32x2_t* p = (const f32x2_t*)(dgp + (int64_t)r * P);
    for (int q = 0; q < P / 2; ++q) {
      const f32x2_t v = p[q];
      s += v[0];
      s += v[1];
    }
  }
  return s;
}

// With dgp set (and k <= h / V), thread c < k of token i also writes the gate
// gradient of the token's slot c, which saves the separate dgate launch.
template <typename T>
__global__ __launch_bounds__(256) void unpermute_kernel(const T* __restrict__ dxp,
                                                        const int32_t* __restrict__ row_of_slot,
                                                        int64_t t0, int tokens, int h, int k,
                                                        T* __restrict__ dX,
                                                        const float* __restrict__ dgp, int P,
                                                        float* __restrict__ dgates) {
  constexpr int V = Elem<T>::kVec;
  const int vpr = h / V;
  const int64_t gid = blockIdx.x * 256ll + threadIdx.x;
  if (gid >= (int64_t)tokens * vpr) return;
  const int i = (int)(gid / vpr), c = (int)(gid % vpr);
  float acc[V];
#pragma unroll
  for (int q = 0; q < V; ++q) acc[q] = 0.f;
  for (int j0 = 0; j0 < k; j0 += 8) {
    int r[8];
    u32x4_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) r[j] = j0 + j < k ? row_of_slot[(int64_t)i * k + j0 + j] : -1;
#pragma unroll
    for (int j = 0; j < 8; ++j)  // (k is uniform: no load past the token's slots;
      if (j0 + j < k)            // a dropped slot, r < 0, reads row 0 and is skipped)
        v[j] = *(const u32x4_t*)(dxp + (int64_t)(r[j] < 0 ? 0 : r[j]) * h + c * V);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (r[j] < 0) continue;
      float f[V];
      unpack16(v[j], f, (T*)nullptr);
#pragma unroll
      for (int q = 0; q < V; ++q) acc[q] += f[q];
    }
  }
  *(u32x4_t*)(dX + (t0 + i) * h + c * V) = pack16(acc, (T*)nullptr);
  if (dgp != nullptr && c < k)
    dgates[(t0 + i) * k + c] = dgate_of_row(dgp, P, row_of_slot[(int64_t)i * k + c]);
}

// One thread per slot of the chunk: dgates[slot] = sum over p of dgp[row][p].
__global__ __launch_bounds__(256) void dgate_kernel(const float* __restrict__ dgp, int P,
                                                    const int32_t* __restrict__ row_of_slot,
                                                    int64_t slot0, int nslots,
                                                    float* __restrict__ dgates) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= nslots) return;
  dgates[slot0 + i] = dgate_of_row(dgp, P, row_of_slot[i]);
}

hipError_t launch_combine(int dtype, const void* y, const int32_t* row_of_slot, const float* gates,
                          int64_t t0, int tokens, int h, int k, void* Y, hipStream_t s) {
  const int V = dtype == 0 ? 8 : 4;
  const int64_t work = (int64_t)tokens * (h / V);
  if (work == 0) return hipSuccess;
  const int blocks = (int)((work + 255) / 256);
  if (dtype == 0)
    combine_kernel<bf16_t><<<blocks, 256, 0, s>>>((const bf16_t*)y, row_of_slot, gates, t0, tokens,
                                                  h, k, (bf16_t*)Y);
  else
    combine_kernel<float><<<blocks, 256, 0, s>>>((const float*)y, row_of_slot, gates, t0, tokens, h,
                                                 k, (float*)Y);
  return hipGetLastError();
}

hipError_t launch_unpermute(int dtype, const void* dxp, const float* dgp, int P,
                            const int32_t* row_of_slot, int64_t t0, int tokens, int h, int k,
                            void* dX, float* dgates, hipStream_t s) {
  const int V = dtype == 0 ? 8 : 4;
  const int64_t work = (int64_t)tokens * (h / V);
  if (work == 0) return hipSuccess;
  const int blocks = (int)((work + 255) / 256);
  const bool fused = k <= h / V;  // every token has a thread per slot
  const float* dgp_f = fused ? dgp : nullptr;
  if (dtype == 0)
    unpermute_kernel<bf16_t><<<blocks, 256, 0, s>>>((const bf16_t*)dxp, row_of_slot, t0, tokens, h,
                                                    k, (bf16_t*)dX, dgp_f, P, dgates);
  else
    unpermute_kernel<float><<<blocks, 256, 0, s>>>((const float*)dxp, row_of_slot, t0, tokens, h, k,
                                                   (float*)dX, dgp_f, P, dgates);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || fused) return err;
  const int nslots = tokens * k;
  dgate_kernel<<<(nslots + 255) / 256, 256, 0, s>>>(dgp, P, row_of_slot, t0 * k, nslots, dgates);
  return hipGetLastError();
}

// ------------------------------------------------ expert-ordered chunks
// The chunk holds rows [p0, p1) of the layer's grouped rows; every token
// reads its k row ids and adds the rows that fall in the chunk, in slot
// order, to an fp32 sum.  The chunk holding the token's first grouped row
// writes the sum; later chunks add it to the stored value (one rounding to
// the storage type per chunk).  A token whose slots are all dropped is
// written as 0 by the first chunk.
constexpr int kNoRow = 0x7fffffff;

template <typename T, bool kGates>
__device__ __forceinline__ void sum_rows_in_chunk(const T* __restrict__ rows,
                                                  const int32_t* __restrict__ row_of_slot,
                                                  const float* __restrict__ gates, int64_t t,
                                                  int h, int k, int c, int p0, int p1,
                                                  float (&acc)[Elem<T>::kVec], bool& any,
                                                  int& rmin) {
  constexpr int V = Elem<T>::kVec;
#pragma unroll
  for (int q = 0; q < V; ++q) acc[q] = 0.f;
  any = false;
  rmin = kNoRow;
  for (int j0 = 0; j0 < k; j0 += 8) {
    int r[8];
    float g[8];
    u32x4_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const bool in = j0 + j < k;
      r[j] = in ? row_of_slot[t * k + j0 + j] : -1;
      g[j] = kGates && in ? gates[t * k + j0 + j] : 1.f;
      if (r[j] >= 0) rmin = min(rmin, r[j]);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (r[j] >= p0 && r[j] < p1) v[j] = *(const u32x4_t*)(rows + (int64_t)(r[j] - p0) * h + c * V);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (!(r[j] >= p0 && r[j] < p1)) continue;
      any = true;
      float f[V];
      unpack16(v[j], f, (T*)nullptr);
#pragma unroll
      for (int q = 0; q < V; ++q) acc[q] = kGates ? fmaf(g[j], f[q], acc[q]) : acc[q] + f[q];
    }
  }
}

// out[t] = sum (first chunk of the token) or out[t] + sum (later chunks)
template <typename T>
__device__ __forceinline__ void store_chunk_sum(T* __restrict__ out, int64_t t, int h, int c,
                                                float (&acc)[Elem<T>::kVec], bool any, int rmin,
                                                int p0, int p1) {
  constexpr int V = Elem<T>::kVec;
  const bool first = (rmin >= p0 && rmin < p1) || (rmin == kNoRow && p0 == 0);
  if (!any && !first) return;
  u32x4_t* o = (u32x4_t*)(out + t * h + c * V);
  if (!first) {
    float f[V];
    unpack16(*o, f, (T*)nullptr);
#pragma unroll
    for (int q = 0; q < V; ++q) acc[q] = f[q] + acc[q];
  }
  *o = pack16(acc, (T*)nullptr);
}

template <typename T>
__global__ __launch_bounds__(256) void combine_rows_kernel(const T* __restrict__ y,
                                                           const int32_t* __restrict__ row_of_slot,
                                                           const float* __restrict__ gates,
                                                           int64_t tokens, int h, int k, int p0,
                                                           int p1, T* __restrict__ Y) {
  constexpr int V = Elem<T>::kVec;
  const int vpr = h / V;
  const int64_t gid = blockIdx.x * 256ll + threadIdx.x;
  if (gid >= tokens * vpr) return;
  const int64_t t = gid / vpr;
  const int c = (int)(gid % vpr);
  float acc[V];
  bool any;
  int rmin;
  sum_rows_in_chunk<T, true>(y, row_of_slot, gates, t, h, k, c, p0, p1, acc, any, rmin);
  store_chunk_sum<T>(Y, t, h, c, acc, any, rmin, p0, p1);
}

// dgates of slot j of token t, when its row is in the chunk (or it is dropped
// and this is the first chunk)
__device__ __forceinline__ void dgate_in_chunk(const float* __restrict__ dgp, int P, int r,
                                               int p0, int p1, float* __restrict__ dst) {
  if (r >= p0 && r < p1) *dst = dgate_of_row(dgp, P, r - p0);
  else if (r < 0 && p0 == 0) *dst = 0.f;
}

template <typename T>
__global__ __launch_bounds__(256) void unpermute_rows_kernel(
    const T* __restrict__ dxp, const int32_t* __restrict__ row_of_slot, int64_t tokens, int h,
    int k, int p0, int p1, T* __restrict__ dX, const float* __restrict__ dgp, int P,
    float* __restrict__ dgates) {
  constexpr int V = Elem<T>::kVec;
  const int vpr = h / V;
  const int64_t gid = blockIdx.x * 256ll + threadIdx.x;
  if (gid >= tokens * vpr) return;
  const int64_t t = gid / vpr;
  const int c = (int)(gid % vpr);
  float acc[V];
  bool any;
  int rmin;
  sum_rows_in_chunk<T, false>(dxp, row_of_slot, nullptr, t, h, k, c, p0, p1, acc, any, rmin);
  store_chunk_sum<T>(dX, t, h, c, acc, any, rmin, p0, p1);
  if (dgp != nullptr && c < k) dgate_in_chunk(dgp, P, row_of_slot[t * k + c], p0, p1, dgates + t * k + c);
}

__global__ __launch_bounds__(256) void dgate_rows_kernel(const float* __restrict__ dgp, int P,
                                                         const int32_t* __restrict__ row_of_slot,
                                                         int64_t nslots, int p0, int p1,
                                                         float* __restrict__ dgates) {
  const int64_t i = blockIdx.x * 256ll + threadIdx.x;
  if (i >= nslots) return;
  dgate_in_chunk(dgp, P, row_of_slot[i], p0, p1, dgates + i);
}

hipError_t launch_combine_rows(int dtype, const void* y, const int32_t* row_of_slot,
                               const float* gates, int64_t T, int h, int k, int p0, int p1, void* Y,
                               hipStream_t s) {
  const int V = dtype == 0 ? 8 : 4;
  const int64_t work = T * (h / V);
  if (work == 0) return hipSuccess;
  const int64_t blocks = (work + 255) / 256;
  if (dtype == 0)
    combine_rows_kernel<bf16_t><<<blocks, 256, 0, s>>>((const bf16_t*)y, row_of_slot, gates, T, h,
                                                       k, p0, p1, (bf16_t*)Y);
  else
    combine_rows_kernel<float><<<blocks, 256, 0, s>>>((const float*)y, row_of_slot, gates, T, h, k,
                                                      p0, p1, (float*)Y);
  return hipGetLastError();
}

hipError_t launch_unpermute_rows(int dtype, const void* dxp, const float* dgp, int P,
                                 const int32_t* row_of_slot, int64_t T, int h, int k, int p0,
                                 int p1, void* dX, float* dgates, hipStream_t s) {
  const int V = dtype == 0 ? 8 : 4;
  const int64_t work = T * (h / V);
  if (work == 0) return hipSuccess;
  const int64_t blocks = (work + 255) / 256;
  const bool fused = k <= h / V;  // every token has a thread per slot
  const float* dgp_f = fused ? dgp : nullptr;
  if (dtype == 0)
    unpermute_rows_kernel<bf16_t><<<blocks, 256, 0, s>>>((const bf16_t*)dxp, row_of_slot, T, h, k,
                                                         p0, p1, (bf16_t*)dX, dgp_f, P, dgates);
  else
    unpermute_rows_kernel<float><<<blocks, 256, 0, s>>>((const float*)dxp, row_of_slot, T, h, k,
                                                        p0, p1, (float*)dX, dgp_f, P, dgates);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || fused) return err;
  const int64_t nslots = T * k;
  dgate_rows_kernel<<<(nslots + 255) / 256, 256, 0, s>>>(dgp, P, row_of_slot, nslots, p0, p1,
                                                         dgates);
  return hipGetLastError();
}

}  // namespace memfine
