// Dispatch kernels: expert histogram, prefix scan and the stable grouping of
// a chunk's token-slots by local expert (the "dispatch" of the paper's
// Eq. (4); the whole-layer histogram is the received-slot count that the
// paper's Section 4.2 "first notification" delivers).
//
// The grouping is deterministic and stable without atomics on output
// cursors: each workgroup owns a fixed, ordered range of slots; a first pass
// counts experts per workgroup, a scan turns the (expert, workgroup) counts
// into first output rows (a single-workgroup kernel, or, while there are few
// counts, each workgroup of the second pass for itself), and a second pass ranks
// the slots of each workgroup in order with wavefront ballots (the set of
// lanes holding the same expert id is found bit by bit) and per-wave counts
// in LDS.
#include "common.h"
#include "kernels.h"

namespace memfine {

__global__ void fill_i32_kernel(int32_t* __restrict__ p, int64_t n, int32_t v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// work[e] += #slots with id e; work[E] += #ids outside [0, E).
__global__ __launch_bounds__(256) void count_kernel(const int32_t* __restrict__ idx, int64_t nslots,
                                                    int E, int32_t* __restrict__ work) {
  extern __shared__ int32_t hist[];
  for (int i = threadIdx.x; i <= E; i += blockDim.x) hist[i] = 0;
  __syncthreads();
  for (int64_t s = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; s < nslots;
       s += (int64_t)gridDim.x * blockDim.x) {
    const int e = idx[s];
    atomicAdd(&hist[((unsigned)e < (unsigned)E) ? e : E], 1);
  }
  __syncthreads();
  for (int i = threadIdx.x; i <= E; i += blockDim.x)
    if (hist[i]) atomicAdd(&work[i], hist[i]);
}

// bcount[e * nb + b] = #slots of expert e in workgroup b's slot range.
__global__ __launch_bounds__(256) void block_hist_kernel(const int32_t* __restrict__ idx, int n,
                                                         int E, int nb, int spb,
                                                         int32_t* __restrict__ bcount) {
  extern __shared__ int32_t hist[];
  for (int e = threadIdx.x; e < E; e += blockDim.x) hist[e] = 0;
  __syncthreads();
  const int s0 = blockIdx.x * spb;
  const int s1 = min(n, s0 + spb);
  for (int s = s0 + threadIdx.x; s < s1; s += blockDim.x) {
    const int e = idx[s];
    if ((unsigned)e < (unsigned)E) atomicAdd(&hist[e], 1);  // ids outside [0,E) are dropped
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x) bcount[(int64_t)e * nb + blockIdx.x] = hist[e];
}

// One workgroup of 1024 threads.  bstart = exclusive scan of bcount in
// expert-major order; counts, offsets (exclusive scan of counts, offsets[E] =
// their total) and order (experts by descending count, ties by id).
__global__ __launch_bounds__(1024) void scan_kernel(const int32_t* __restrict__ bcount, int E,
                                                    int nb, int n, int32_t* __restrict__ bstart,
                                                    int32_t* __restrict__ counts,
                                                    int32_t* __restrict__ offsets,
                                                    int32_t* __restrict__ order) {
  __shared__ int32_t part[1024];
  __shared__ int32_t cnt[1024];
  const int tid = threadIdx.x;
  const int64_t m = (int64_t)E * nb;
  const int64_t per = (m + 1023) / 1024;
  const int64_t b0 = min(m, tid * per), b1 = min(m, b0 + per);
  int32_t sum = 0;
  for (int64_t i = b0; i < b1; ++i) sum += bcount[i];
  part[tid] = sum;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int32_t v = tid >= off ? part[tid - off] : 0;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  int32_t run = part[tid] - sum;
  for (int64_t i = b0; i < b1; ++i) {
    bstart[i] = run;
    run += bcount[i];
  }
  // expert e's rows start where its first workgroup's rows start (the scan
  // is expert-major), so offsets and counts follow from bstart at the
  // expert boundaries; offsets[E] is the total (ids outside [0, E) dropped)
  __syncthreads();
  const int32_t total = part[1023];
  for (int e = tid; e < E; e += 1024) {
    const int32_t o0 = nb > 0 ? bstart[(int64_t)e * nb] : 0;
    const int32_t o1 = e + 1 < E ? (nb > 0 ? bstart[(int64_t)(e + 1) * nb] : 0) : total;
    offsets[e] = o0;
    counts[e] = o1 - o0;
    cnt[e] = o1 - o0;
  }
  if (tid == 0) offsets[E] = total;
  __syncthreads();
  // order: experts by descending count, ties by id
  for (int e = tid; e < E; e += 1024) {
    const int32_t c = cnt[e];
    int rank = 0;
    for (int e2 = 0; e2 < E; ++e2) rank += (cnt[e2] > c) || (cnt[e2] == c && e2 < e);
    order[rank] = e;
  }
}

// Exclusive scan over v[0..m) in place (one workgroup of 256 threads, m any
// size): each thread scans a contiguous run, the run totals are scanned in
// LDS, then each run is offset.  `part` is 256 ints of LDS.  Returns the total.
__device__ int32_t block_exclusive_scan(int32_t* v, int m, int32_t* part) {
  const int tid = threadIdx.x, per = (m + 255) / 256;
  const int a = min(m, tid * per), b = min(m, a + per);
  int32_t sum = 0;
  for (int i = a; i < b; ++i) sum += v[i];
  part[tid] = sum;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    const int32_t x = tid >= off ? part[tid - off] : 0;
    __syncthreads();
    part[tid] += x;
    __syncthreads();
  }
  int32_t run = part[tid] - sum;
  const int32_t total = part[255];
  for (int i = a; i < b; ++i) {
    const int32_t x = v[i];
    v[i] = run;
    run += x;
  }
  __syncthreads();
  return total;
}

// Stable scatter (an id outside [0, E) - which memfine_count reports - is
// dropped: it gets no row and row_of_slot = -1).  Workgroup b walks its slot
// range in rounds of 256 slots (4 waves x 64 lanes, in slot order; with 256
// slots per workgroup that is one round, so a chunk's slots spread over
// n / 256 workgroups).  A lane's output row is
//   first row of (expert, b) + slots of that expert in earlier rounds
//   + slots of that expert in earlier waves of this round + its rank among
//   the lanes of its own wave holding the same expert.
//
// kFused: the workgroup derives its first rows from the per-block counts
// itself (the total of every expert over all blocks, scanned over experts,
// plus the expert's slots in earlier blocks), and workgroup 0 writes counts,
// offsets and order, which saves the single-workgroup scan launch; used
// while E * nb is small enough that every workgroup reading all counts is
// cheap.
template <bool kFused>
__global__ __launch_bounds__(256) void scatter_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ gates, int n, int E, int k,
    int slot0, int nb, int spb, const int32_t* __restrict__ bstart, int32_t* __restrict__ sorted_slot,
    int32_t* __restrict__ row_of_slot, int32_t* __restrict__ tok_of_row,
    float* __restrict__ gate_of_row, const int32_t* __restrict__ bcount,
    int32_t* __restrict__ counts, int32_t* __restrict__ offsets, int32_t* __restrict__ order) {
  extern __shared__ int32_t sh[];
  int32_t* run = sh;      // [E]     next row per expert for this workgroup
  int32_t* wc = sh + E;   // [4][E]  per-wave counts of the current round
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if constexpr (kFused) {
    int32_t* tot = wc;           // [E] slots of each expert in the chunk, then its first row
    int32_t* pre = wc + E;       // [E] the expert's slots in the workgroups before this one
    int32_t* cnt = wc + 2 * E;   // [E] the counts, kept for the order
    __shared__ int32_t spart[256];
    for (int e = tid; e < E; e += 256) tot[e] = pre[e] = 0;
    __syncthreads();
    const int64_t m = (int64_t)E * nb;
    for (int64_t i = tid; i < m; i += 256) {
      const int32_t v = bcount[i];
      if (v) {
        const int e = (int)(i / nb), b = (int)(i % nb);
        atomicAdd(&tot[e], v);
        if (b < (int)blockIdx.x) atomicAdd(&pre[e], v);
      }
    }
    __syncthreads();
    for (int e = tid; e < E; e += 256) cnt[e] = tot[e];
    __syncthreads();
    const int32_t total = block_exclusive_scan(tot, E, spart);
    for (int e = tid; e < E; e += 256) run[e] = tot[e] + pre[e];
    if (blockIdx.x == 0) {
      for (int e = tid; e < E; e += 256) {
        counts[e] = cnt[e];
        offsets[e] = tot[e];
        // order: experts by descending count, ties by id
        const int32_t c = cnt[e];
        int rank = 0;
        for (int e2 = 0; e2 < E; ++e2) rank += (cnt[e2] > c) || (cnt[e2] == c && e2 < e);
        order[rank] = e;
      }
      if (tid == 0) offsets[E] = total;
    }
    __syncthreads();
  } else {
    for (int e = tid; e < E; e += 256) run[e] = bstart[(int64_t)e * nb + blockIdx.x];
  }
  for (int i = tid; i < 4 * E; i += 256) wc[i] = 0;
  __syncthreads();
  const int nbits = E > 1 ? 32 - __clz(E - 1) : 0;
  const int s0 = blockIdx.x * spb;
  const int s1 = min(n, s0 + spb);
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int base = s0; base < s1; base += 256) {
    const int s = base + tid;
    const int e_raw = s < s1 ? idx[s] : 0;
    const bool valid = s < s1 && (unsigned)e_raw < (unsigned)E;
    const int e = valid ? e_raw : 0;
    if (s < s1 && !valid) row_of_slot[s] = -1;  // dropped slot: no row
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < nbits; ++b) {
      const bool bit = (e >> b) & 1;
      const uint64_t m = __ballot(valid && bit);
      peers &= bit ? m : ~m;
    }
    const int rank = __popcll(peers & below);
    if (valid && rank == 0) wc[w * E + e] = __popcll(peers);
    __syncthreads();
    if (valid) {
      int pos = run[e] + rank;
      for (int w2 = 0; w2 < w; ++w2) pos += wc[w2 * E + e];
      const int gs = slot0 + s;
      sorted_slot[pos] = gs;
      row_of_slot[s] = pos;
      tok_of_row[pos] = gs / k;
      if (gates) gate_of_row[pos] = gates[s];
    }
    __syncthreads();
    for (int e2 = tid; e2 < E; e2 += 256) {
      run[e2] += wc[e2] + wc[E + e2] + wc[2 * E + e2] + wc[3 * E + e2];
      wc[e2] = wc[E + e2] = wc[2 * E + e2] = wc[3 * E + e2] = 0;
    }
    __syncthreads();
  }
}

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int blocks = (int)std::min<int64_t>((n + 255) / 256, 1024);
  fill_i32_kernel<<<blocks, 256, 0, s>>>(p, n, v);
  return hipGetLastError();
}

hipError_t launch_count(const int32_t* idx, int64_t nslots, int E, int32_t* work, hipStream_t s) {
  hipError_t err = launch_fill_i32(work, E + 1, 0, s);
  if (err != hipSuccess || nslots == 0) return err;
  const int blocks = (int)std::min<int64_t>((nslots + 255) / 256, 1024);
  count_kernel<<<blocks, 256, (E + 1) * sizeof(int32_t), s>>>(idx, nslots, E, work);
  return hipGetLastError();
}

hipError_t launch_dispatch(const int32_t* idx, const float* gates, int64_t slot0, int n, int E,
                           int k, const ChunkMeta& m, hipStream_t s) {
  const int nb = dispatch_blocks(n), spb = dispatch_slots_per_block(n);
  const int32_t* cidx = idx + slot0;
  if (nb > 0) {
    block_hist_kernel<<<nb, 256, E * sizeof(int32_t), s>>>(cidx, n, E, nb, spb, m.bcount);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  // small E x nb: the scatter workgroups scan the counts themselves
  const bool fused = nb > 0 && (int64_t)E * nb <= 16384;
  if (!fused) {
    scan_kernel<<<1, 1024, 0, s>>>(m.bcount, E, nb, n, m.bstart, m.counts, m.offsets, m.order);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess || nb == 0) return err;
    scatter_kernel<false><<<nb, 256, 5 * E * sizeof(int32_t), s>>>(
        cidx, gates ? gates + slot0 : nullptr, n, E, k, (int)slot0, nb, spb, m.bstart,
        m.sorted_slot, m.row_of_slot, m.tok_of_row, m.gate_of_row, nullptr, nullptr, nullptr,
        nullptr);
  } else {
    scatter_kernel<true><<<nb, 256, 5 * E * sizeof(int32_t), s>>>(
        cidx, gates ? gates + slot0 : nullptr, n, E, k, (int)slot0, nb, spb, m.bstart,
        m.sorted_slot, m.row_of_slot, m.tok_of_row, m.gate_of_row, m.bcount, m.counts, m.offsets,
        m.order);
  }
  return hipGetLastError();
}

// The view of an expert-ordered chunk, rows [p0, p1) of the layer's grouped
// rows: one thread per expert (E <= 1024).  The experts that get a weight-
// gradient tile (mode != 0) come first in order_c, by descending row count
// in the chunk (ties: lower id), then the rest by id.
__global__ __launch_bounds__(1024) void chunk_view_kernel(
    const int32_t* __restrict__ offsets, int E, int p0, int p1, int first, int accumulate,
    int32_t* __restrict__ offsets_c, int32_t* __restrict__ order_c,
    int32_t* __restrict__ wexperts, int32_t* __restrict__ wmode) {
  __shared__ int32_t key[1024];
  __shared__ int32_t n_tiles;
  const int e = threadIdx.x;
  if (e == 0) n_tiles = 0;
  __syncthreads();
  int k = -1;
  if (e < E) {
    const int lo = offsets[e], hi = offsets[e + 1];
    const int a = min(max(lo, p0), p1), b = min(max(hi, p0), p1);
    offsets_c[e] = a - p0;
    if (e == E - 1) offsets_c[E] = b - p0;
    const int rows = b - a;
    int m;
    if (rows > 0) m = (!accumulate && lo >= p0) ? 1 : 2;  // the expert's first rows: overwrite
    else m = (lo == hi && first && !accumulate) ? 1 : 0;  // no rows at all: zeros, once
    wmode[e] = m;
    if (m != 0) atomicAdd(&n_tiles, 1);
    k = m != 0 ? rows : -1;  // sort key: experts without a tile last
    key[e] = k;
  }
  __syncthreads();
  if (e < E) {
    int rank = 0;
    for (int q = 0; q < E; ++q) {
      const int kq = key[q];
      rank += (kq > k) || (kq == k && q < e);
    }
    order_c[rank] = e;
  }
  if (e == 0) *wexperts = n_tiles;
}

hipError_t launch_chunk_view(const int32_t* offsets, int E, int p0, int p1, int first,
                             int accumulate, int32_t* offsets_c, int32_t* order_c,
                             int32_t* wexperts, int32_t* wmode, hipStream_t s) {
  if (E < 1 || E > 1024) return hipErrorInvalidValue;
  chunk_view_kernel<<<1, 1024, 0, s>>>(offsets, E, p0, p1, first, accumulate, offsets_c, order_c,
                                       wexperts, wmode);
  return hipGetLastError();
}

}  // namespace memfine
