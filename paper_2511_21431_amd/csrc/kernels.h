// Host-side launchers of the gfx950 kernels (internal to libmemfine).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace memfine {

// Slots handled by one workgroup of the dispatch histogram / scatter kernels:
// 256 (one round of the scatter) while that needs at most 128 workgroups,
// else the smallest power-of-two multiple that does, which bounds the
// per-workgroup count tables at E * 128 entries.  Every scatter workgroup
// reads all E x nb block counts for its prefix: at 131072 slots, 512
// workgroups of 256 slots spent most of the dispatch's 57 us on that read;
// 128 of 1024 take 25 us.
inline int dispatch_slots_per_block(int64_t n) {
  int64_t spb = 256;
  while ((n + spb - 1) / spb > 128) spb *= 2;
  return (int)spb;
}
inline int dispatch_blocks(int64_t n) {
  const int spb = dispatch_slots_per_block(n);
  return (int)((n + spb - 1) / spb);
}

// Per-chunk routing metadata produced by the dispatch kernels; all device.
struct ChunkMeta {
  int32_t* bcount;       // [E * nb]  per-workgroup expert histograms (expert-major)
  int32_t* bstart;       // [E * nb]  their exclusive scan = first output row
  int32_t* counts;       // [E]
  int32_t* offsets;      // [E + 1]
  int32_t* order;        // [E]       experts by descending count (ties: lower id)
  int32_t* sorted_slot;  // [n]       global slot id of each grouped row
  int32_t* row_of_slot;  // [n]       grouped row of the chunk's i-th slot
  int32_t* tok_of_row;   // [n]       token of each grouped row
  float* gate_of_row;    // [n]       gate of each grouped row
};

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s);
hipError_t launch_count(const int32_t* idx, int64_t nslots, int E, int32_t* work, hipStream_t s);
// Dispatch of slots [slot0, slot0 + n) of the flat idx array (one chunk).
hipError_t launch_dispatch(const int32_t* idx, const float* gates, int64_t slot0, int n, int E,
                           int k, const ChunkMeta& m, hipStream_t s);

// Expert-ordered chunks: chunk c is rows [p0, p1) of the layer's slots
// grouped by expert (one dispatch over all tokens).  From the layer's
// offsets [E + 1], the chunk's view: its offsets [E + 1] (rows relative to
// p0), its experts with a weight-gradient tile first, by descending row
// count [E], their number [1], and each expert's weight-gradient mode [E]
// (0: no tile, 1: overwrite dW, 2: add to dW).  `first`: the first chunk
// (overwrites the dW of experts without rows unless `accumulate`).
hipError_t launch_chunk_view(const int32_t* offsets, int E, int p0, int p1, int first,
                             int accumulate, int32_t* offsets_c, int32_t* order_c,
                             int32_t* wexperts, int32_t* wmode, hipStream_t s);

// Gate-weighted combine, Y[t0 + i] = sum_j g[t, j] * y[row_of_slot[i*k + j]].
hipError_t launch_combine(int dtype, const void* y, const int32_t* row_of_slot, const float* gates,
                          int64_t t0, int tokens, int h, int k, void* Y, hipStream_t s);
// dX[t0 + i] = sum_j dxp[row_of_slot[i*k + j]];  dgates[t, j] = sum_p dgp[row][p].
hipError_t launch_unpermute(int dtype, const void* dxp, const float* dgp, int P,
                            const int32_t* row_of_slot, int64_t t0, int tokens, int h, int k,
                            void* dX, float* dgates, hipStream_t s);

// The same over all T tokens for an expert-ordered chunk, rows [p0, p1) of
// the layer's grouped rows (y and dxp hold those rows, from row p0): each
// token adds its slots in the chunk to Y (dX), and the chunk that holds its
// first grouped row overwrites instead (the first chunk, for a token whose
// slots are all dropped).  dgates of the chunk's slots are written.
hipError_t launch_combine_rows(int dtype, const void* y, const int32_t* row_of_slot,
                               const float* gates, int64_t T, int h, int k, int p0, int p1, void* Y,
                               hipStream_t s);
hipError_t launch_unpermute_rows(int dtype, const void* dxp, const float* dgp, int P,
                                 const int32_t* row_of_slot, int64_t T, int h, int k, int p0,
                                 int p1, void* dX, float* dgates, hipStream_t s);

// Grouped GEMMs.  Row-grouped problems: rows [offsets[e], offsets[e+1]) belong
// to expert e.  n is the chunk's slot count (an upper bound for the grid).
struct GemmArgs {
  int dtype;
  int n, E, h, F;
  const int32_t* offsets;
  const int32_t* order;
  const int32_t* tok_of_row;
  const float* gate_of_row;
  const void* X;     // [T, h]
  const void* dY;    // [T, h]
  const void* W1;    // [E, 2F, h]
  const void* W2;    // [E, h, F]
  void* a;           // [n, F]   forward SwiGLU output
  void* y;           // [n, h]   forward expert output
  void* u;           // [n, 2F]  backward: du
  void* ag;          // [n, F]   backward: dA, then gate * SwiGLU output in place
  void* dxp;         // [n, h]   backward: input gradient per row
  float* dgp;        // [n, P]   backward: partial gate gradients
  int P;             // partials per row
  float* dW1;        // [E, 2F, h]
  float* dW2;        // [E, h, F]
  int accumulate;    // wgrad: 1 = add into dW, 0 = overwrite
  const int32_t* wmode;     // wgrad, or null: per expert 0 no tile, 1 overwrite, 2 add
  const int32_t* wexperts;  // wgrad with wmode: experts with a tile (the first of order)
  int64_t T_h_bytes; // bytes of X (and of dY): T * h * element size
  int tile_override; // 0: per problem; 1: 128 x 128; 2: 256 x 256 direct; 3: 256 x 256 staged
  int raster;        // tile order: -1 per problem; 0 row-major; 1..3 XCD blocks, groups of 4/8/16 m-tiles; 4 XCD blocks, row-major
  int cus;           // compute units of the device
  int split_tail;    // 1: row-grouped GEMMs run a short last round as quarter tiles
  int32_t* tile_ctr; // weight gradients: device tile counter (one int) for a dynamic
                     // persistent launch, or null for one tile per workgroup
};

int dgate_partials(int F);

// Router (E <= 256 experts, k <= 16): logits on the matrix cores, softmax,
// top-k and renormalised gates; logits may be null.
hipError_t launch_router_fwd(int dtype, const void* X, const void* Wr, int64_t T, int h, int E,
                             int k, int32_t* idx, float* gates, float* logits, hipStream_t s);
// Router forward in two steps for wide routers: the logits [T, E] (fp32) as a
// grouped GEMM (launch_router_logits: one "expert" of T rows; X in a, K = h
// in F, Wr in W2, E in h, logits in y, offsets {0, T}), then their top-k
// (64 < E <= 256, k <= 16) with the selection and gates of launch_router_fwd.
hipError_t launch_router_logits(const GemmArgs& g, hipStream_t s);
hipError_t launch_router_topk(const float* logits, int64_t T, int E, int k, int32_t* idx,
                              float* gates, hipStream_t s);
// Router backward, per token: the dense dz rows D [T, EP] and, with
// `with_dx`, dX (+)= dz Wr (else launch_router_dx computes it from D).
hipError_t launch_router_bwd_dx(int dtype, const void* Wr, const int32_t* idx, const float* gates,
                                const float* dgates, int64_t T, int h, int E, int k, int EP,
                                int accumulate, int with_dx, void* dX, void* D, hipStream_t s);
// dX (+)= D Wr as a grouped GEMM (E % 64 == 0): one "expert" of T rows; D in
// dY (K = E in h, identity tok_of_row), Wr in W2, the hidden size in F, dX in
// ag, `accumulate` adds to it.
hipError_t launch_router_dx(const GemmArgs& g, hipStream_t s);
// Row ranges of S splits of T rows (offsets [S + 1], order [S]) and the
// identity row -> token table [T], for the split-K weight gradient.
hipError_t launch_router_split_meta(int32_t* offsets, int32_t* order, int32_t* tok, int64_t T, int S,
                                    hipStream_t s);
// dWr (+)= sum over the S partial products P [S, EP, h].
hipError_t launch_router_reduce(const float* P, int S, int EP, int E, int h, int accumulate,
                                float* dWr, hipStream_t s);

hipError_t launch_fc1_fwd(const GemmArgs& g, hipStream_t s);
hipError_t launch_fc2_fwd(const GemmArgs& g, hipStream_t s);
hipError_t launch_fc1_recompute(const GemmArgs& g, hipStream_t s);
hipError_t launch_fc2_dgrad(const GemmArgs& g, hipStream_t s);
hipError_t launch_fc2_wgrad(const GemmArgs& g, hipStream_t s);
hipError_t launch_fc1_wgrad(const GemmArgs& g, hipStream_t s);
hipError_t launch_fc1_dgrad(const GemmArgs& g, hipStream_t s);
// FC1 dgrad and FC1 wgrad in one launch (independent problems).
hipError_t launch_fc1_dgrad_wgrad(const GemmArgs& g, hipStream_t s);

}  // namespace memfine
