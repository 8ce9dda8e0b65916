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

// One workgroup per potential run i of the sorted keys: row i of U is the
// weighted sum, in entry order, of the dy rows of the entries of run i;
// rows past the active ones (and the dropped-entry run) are zero, their row
// id -1.  count[0] = active rows, count[1] = dropped entries.
__global__ __launch_bounds__(kThreads) void emb_segsum_kernel(
    const int32_t* __restrict__ uniq, const int32_t* __restrict__ lens, const int32_t* __restrict__ offs,
    const int32_t* __restrict__ nruns, const int32_t* __restrict__ vals, const int32_t* __restrict__ feat,
    const float* __restrict__ weight, const float* __restrict__ dy, int64_t ld_dy, int dim, int32_t vocab, int nnz,
    int32_t* __restrict__ rows, float* __restrict__ U, int32_t* __restrict__ count) {
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
  float* u = U + (int64_t)i * dim;
  const bool vec = (dim & 3) == 0 && (ld_dy & 3) == 0 && (reinterpret_cast<uintptr_t>(dy) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(U) & 15) == 0;
  if (vec) {
    for (int c = 4 * threadIdx.x; c < dim; c += 4 * kThreads) {
      f4v acc = {0.f, 0.f, 0.f, 0.f};
      if (active) {
        const int t0 = offs[i], t1 = t0 + lens[i];
        for (int t = t0; t < t1; ++t) {
          const int e = vals[t];
          const int f = feat ? feat[e] : e;
          const float w = weight ? weight[e] : 1.f;
          const f4v v = gload<f4v>(dy + (int64_t)f * ld_dy + c);
          acc += w * v;
        }
      }
      gstore<f4v>(u + c, acc);
    }
  } else {
    for (int c = threadIdx.x; c < dim; c += kThreads) {
      float acc = 0.f;
      if (active) {
        const int t0 = offs[i], t1 = t0 + lens[i];
        for (int t = t0; t < t1; ++t) {
          const int e = vals[t];
          const int f = feat ? feat[e] : e;
          const float w = weight ? weight[e] : 1.f;
          acc += w * gload<float>(dy + (int64_t)f * ld_dy + c);
        }
      }
      gstore<float>(u + c, acc);
    }
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
