// Device kernels for embedding layers (appendix "Shampoo for embedding
// layers"): the sparse gradient of a lookup in compact form, and the reduce
// of split-K partial statistics.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"

namespace shp {

// Sort keys of the lookup entries: the table row, or `vocab` (sorts last)
// for an entry whose row or output feature is out of range; values are the
// entry indices, so a stable sort keeps the entries of one row in order.
__global__ __launch_bounds__(kThreads) void emb_keys_kernel(const int32_t* __restrict__ idx,
                                                           const int32_t* __restrict__ feat, int nnz,
                                                           int32_t vocab, int m, int32_t* __restrict__ keys,
                                                           int32_t* __restrict__ vals, int32_t* __restrict__ lens) {
  const int e = blockIdx.x * kThreads + threadIdx.x;
  if (e >= nnz) return;
  const int32_t r = idx[e];
  const int32_t f = feat ? feat[e] : e;
  keys[e] = (r >= 0 && r < vocab && f >= 0 && f < m) ? r : vocab;
  vals[e] = e;
  lens[e] = 0;  // run lengths past the last run stay 0 for the offset scan
}

// Segment sums of the sorted entries in fixed chunks of kEmbChunk entries,
// one workgroup per chunk.  A run (the entries of one table row) that lies
// inside the chunk is summed into its row of U directly; the run holding
// the chunk's first entry, if it reaches outside the chunk, goes to partial
// slot 0 of the chunk, and the chunk's last run, if different and reaching
// past the end, to slot 1.  Entries are added in sorted (= entry) order.
constexpr int kEmbChunk = 64;

template <bool VEC>
__device__ __forceinline__ void emb_chunk_cols(int c, const int32_t* __restrict__ uniq, const int32_t* __restrict__ lens,
                                               const int32_t* __restrict__ offs, int R, const int32_t* __restrict__ vals,
                                               const int32_t* __restrict__ feat, const float* __restrict__ weight,
                                               const float* __restrict__ dy, int64_t ld_dy, int dim, int32_t vocab,
                                               int nnz, float* __restrict__ U, float* __restrict__ part) {
  const int t0 = c * kEmbChunk, t1 = min(t0 + kEmbChunk, nnz);
  // run holding t0: the last run starting at or before t0
  int lo = 0, hi = R - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (offs[mid] <= t0) lo = mid; else hi = mid - 1;
  }
  constexpr int W = VEC ? 4 : 1;
  for (int col = W * threadIdx.x; col < dim; col += W * kThreads) {
    int i = lo;
    int rs = offs[i], re = rs + lens[i];
    bool skip = uniq[i] == vocab;
    f4v acc = {0.f, 0.f, 0.f, 0.f};
    auto flush = [&]() {
      if (skip) return;
      float* dst;
      if (rs >= t0 && re <= t1) dst = U + (int64_t)i * dim;              // whole run in this chunk
      else if (i == lo) dst = part + ((int64_t)c * 2 + 0) * dim;         // run of the first entry
      else dst = part + ((int64_t)c * 2 + 1) * dim;                      // last run, continues
      if (VEC) gstore<f4v>(dst + col, acc);
      else gstore<float>(dst + col, acc[0]);
    };
    for (int t = t0; t < t1; ++t) {
      if (t >= re) {
        flush();
        ++i;
        rs = offs[i];
        re = rs + lens[i];
        skip = uniq[i] == vocab;
        acc = f4v{0.f, 0.f, 0.f, 0.f};
      }
      if (skip) continue;
      const int e = vals[t];
      const int f = feat ? feat[e] : e;
      const float w = weight ? weight[e] : 1.f;
      const float* src = dy + (int64_t)f * ld_dy + col;
      if (VEC) acc += w * gload<f4v>(src);
      else acc[0] += w * gload<float>(src);
    }
    flush();
  }
}

__global__ __launch_bounds__(kThreads) void emb_chunk_kernel(
    const int32_t* __restrict__ uniq, const int32_t* __restrict__ lens, const int32_t* __restrict__ offs,
    const int32_t* __restrict__ nruns, const int32_t* __restrict__ vals, const int32_t* __restrict__ feat,
    const float* __restrict__ weight, const float* __restrict__ dy, int64_t ld_dy, int dim, int32_t vocab, int nnz,
    float* __restrict__ U, float* __restrict__ part) {
  const int c = blockIdx.x;
  if (c * kEmbChunk >= nnz) return;
  const int R = *nruns;
  if (R < 1) return;
  const bool vec = (dim & 3) == 0 && (ld_dy & 3) == 0 && (reinterpret_cast<uintptr_t>(dy) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(U) & 15) == 0;
  if (vec) emb_chunk_cols<true>(c, uniq, lens, offs, R, vals, feat, weight, dy, ld_dy, dim, vocab, nnz, U, part);
  else emb_chunk_cols<false>(c, uniq, lens, offs, R, vals, feat, weight, dy, ld_dy, dim, vocab, nnz, U, part);
}

// One workgroup per potential run i: the row id (-1 past the active rows),
// the counts (count[0] = active rows, count[1] = dropped entries), and for a
// run that spans several chunks the sum of its chunk partials in chunk
// order.  Rows of U at or past the active count are not written.
__global__ __launch_bounds__(kThreads) void emb_fix_kernel(const int32_t* __restrict__ uniq,
                                                          const int32_t* __restrict__ lens,
                                                          const int32_t* __restrict__ offs,
                                                          const int32_t* __restrict__ nruns, int dim, int32_t vocab,
                                                          int nnz, const float* __restrict__ part,
                                                          int32_t* __restrict__ rows, float* __restrict__ U,
                                                          int32_t* __restrict__ count) {
  const int i = blockIdx.x;
  if (i >= nnz) return;
  const int R = *nruns;
  const bool tail_dropped = R > 0 && uniq[R - 1] == vocab;
  if (i == 0 && threadIdx.x == 0) {
    count[0] = R - (tail_dropped ? 1 : 0);
    count[1] = tail_dropped ? lens[R - 1] : 0;
  }
  const bool active = i < R && uniq[i] != vocab;
  if (threadIdx.x == 0) rows[i] = active ? uniq[i] : -1;
  if (!active) return;
  const int rs = offs[i], re = rs + lens[i];
  const int c0 = rs / kEmbChunk, c1 = (re - 1) / kEmbChunk;
  if (c0 == c1) return;  // summed in place by its chunk
  for (int col = threadIdx.x; col < dim; col += kThreads) {
    float acc = 0.f;
    for (int c = c0; c <= c1; ++c) {
      const int slot = (c == c0 && rs != c0 * kEmbChunk) ? 1 : 0;
      acc += gload<float>(part + ((int64_t)c * 2 + slot) * dim + col);
    }
    gstore<float>(U + (int64_t)i * dim + col, acc);
  }
}

// R = beta R + alpha * sum_s part[s] over all n elements, the partials added
// in split order (deterministic).  beta == 1 keeps R's old value exactly
// scaled by one.
__global__ __launch_bounds__(kThreads) void emb_reduce_kernel(const float* __restrict__ part, int splits,
                                                             int64_t stride, int64_t n, float alpha, float beta,
                                                             float* __restrict__ R) {
  const int64_t q = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * 4;
  if (q >= n) return;
  if (q + 4 <= n && (n & 3) == 0) {
    f4v acc = {0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < splits; ++s) acc += gload<f4v>(part + s * stride + q);
    f4v r = gload<f4v>(R + q);
    gstore<f4v>(R + q, beta * r + alpha * acc);
  } else {
    for (int64_t k = q; k < q + 4 && k < n; ++k) {
      float acc = 0.f;
      for (int s = 0; s < splits; ++s) acc += gload<float>(part + s * stride + k);
      gstore<float>(R + k, beta * gload<float>(R + k) + alpha * acc);
    }
  }
}

}  // namespace shp
