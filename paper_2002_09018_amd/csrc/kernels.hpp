// Device kernels of the Shampoo hot path (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <type_traits>

#include "tile_mfma.hpp"

#ifndef SHP_EPI_VEC
#define SHP_EPI_VEC 1
#endif

namespace shp {

typedef float f4v __attribute__((ext_vector_type(4)));

// Sum over the workgroup (fixed order: waves, then the per-wave partials).
__device__ __forceinline__ double block_sum(double v, double* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int w = 0; w < kThreads / 64; ++w) s += red[w];
  return s;
}

template <typename SG>
__device__ __forceinline__ float load_g(const void* G, int64_t i) {
  return cvt<float, SG>(reinterpret_cast<const SG*>(G)[i]);
}

// D^{-1/2} o G with 0 where D == 0.
__device__ __forceinline__ float ada_dir(float g, float d) { return d > 0.f ? g / sqrtf(d) : 0.f; }

// Element access of the graft passes: 4 consecutive elements of a row.
template <typename SG>
struct G4;
template <>
struct G4<float> {
  static __device__ __forceinline__ void load(const void* G, int64_t i, float g[4]) {
    typedef float f4 __attribute__((ext_vector_type(4)));
    const f4 v = gload<f4>(reinterpret_cast<const float*>(G) + i);
    g[0] = v[0]; g[1] = v[1]; g[2] = v[2]; g[3] = v[3];
  }
};
template <>
struct G4<uint16_t> {
  static __device__ __forceinline__ void load(const void* G, int64_t i, float g[4]) {
    typedef uint16_t u4 __attribute__((ext_vector_type(4)));
    const u4 v = gload<u4>(reinterpret_cast<const uint16_t*>(G) + i);
    g[0] = cvt<float, uint16_t>(v[0]); g[1] = cvt<float, uint16_t>(v[1]);
    g[2] = cvt<float, uint16_t>(v[2]); g[3] = cvt<float, uint16_t>(v[3]);
  }
};


// ============================================================================
// Grouped GEMM for statistics and preconditioning.
// One "problem" per output matrix; workgroups enumerate the 128 x 128 output
// tiles of all problems (only the upper-triangular tiles of a symmetric
// output, whose tiles are mirrored).
//   C = alpha * opA(A) opB(B) + beta * C      (beta == 0: C is not read)
// ============================================================================
struct GemmProblem {
  const void* A;
  const void* B;
  float* C;
  int64_t lda, ldb, ldc;
  int a_rows, a_cols;  // A as stored
  int b_rows, b_cols;  // B as stored
  int M, N, K;
  float alpha, beta;
  int sym;        // symmetric output: compute tiles ti <= tj, mirror into the lower part
  int tiles_n;    // ceil(N / 128)
  int tile_begin; // first logical tile of this problem
  int a_aligned, b_aligned;
  // Optional device-side limits (embedding rows, whose count is known only
  // on the device), honoured by the LIM instantiation:
  //   ksplit == 0: K is cut to *kcount - koff (>= 0);
  //   ksplit  > 0: split koff of ksplit equal parts of the first *kcount
  //                k-indices (parts rounded up to the 16-deep k stage);
  // the k-extent of the operands is cut with K; tiles starting at or past
  // row *mcount are skipped.
  const int* kcount;
  const int* mcount;
  int koff, ksplit;
  // Graft pass 1 fused into the preconditioning GEMM that writes P (graft
  // instantiation, gD != NULL): for every output element (r, c),
  // D = D + G o G, and per output tile the sums of (D^{-1/2} o G)^2 and P^2
  // into gpart[2 (part_base + tile)] and gpart[2 (part_base + tile) + 1].
  // G and D are the block's views (row stride ldg, the same as P's).
  const void* gG;
  float* gD;
  int64_t ldg;
  double* gpart;
  int part_base;
};

__device__ __forceinline__ int find_problem_gemm(const GemmProblem* probs, int nprob, int t) {
  int lo = 0, hi = nprob - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (probs[mid].tile_begin <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Epilogue row stores: a wave's MFMA block row (kM rows x 64 columns, laid
// out row-major in `epi` by the caller) goes out as 16-byte row segments
// instead of the accumulators' column-wise 4-byte stores.  `epi` is the
// wave's own slice of the (then unused) stage buffers, so only the wave's
// own LDS ordering is involved.
__device__ __forceinline__ void epi_rows(const float* epi, float* dst, int64_t ld, int lane) {
  constexpr int kM = Mfma<float>::kM;
  constexpr int kSeg = kWaveTile / 4;  // 16-byte segments per row
#pragma unroll
  for (int k = 0; k < kM * kSeg / 64; ++k) {
    const int idx = lane + 64 * k, rr = idx / kSeg, c4 = (idx % kSeg) * 4;
    gstore<f4v>(dst + (int64_t)rr * ld + c4, *reinterpret_cast<const f4v*>(epi + rr * kWaveTile + c4));
  }
}

// LIM: honour the device-side limits kcount / mcount (a separate
// instantiation, so the plain kernels carry no extra registers).
// SGG (not void): element type of G for the fused graft pass 1 (problems
// with gD set; a separate instantiation as well).
// WN = 2: 128 x 256 output tiles (plain outputs, both operands k-major;
// tiles_n counts 256-wide tile columns).
// map: how workgroups find their tiles (kMapXcd, kMapDeal, kMapDiagLast).
template <typename SA, int LA, typename SB, int LB, bool LIM = false, typename SGG = void, int WN = 1>
__global__ __launch_bounds__(kThreads, kMinWaves) void gemm_grouped_kernel(const GemmProblem* __restrict__ probs,
                                                               int nprob, int total_tiles, int map) {
  static_assert(WN == 1 || (!LIM && LA == kLayoutK && LB == kLayoutK), "wide tiles: plain k-major products");
  constexpr int TN = kTile * WN;  // output tile width
  __shared__ __attribute__((aligned(16))) float sa0[StageElems<float, LA>::value], sa1[StageElems<float, LA>::value];
  __shared__ __attribute__((aligned(16))) float sb0[StageElems<float, LB, TN>::value],
      sb1[StageElems<float, LB, TN>::value];
  // LIM: work depends on device-side counts and sits in the first logical
  // tiles; dispatch order (round robin over the XCDs) spreads it evenly.
  int pi, ti, tj, lt = 0;  // lt: the tile's index in its problem (graft partial slots)
  if (!LIM && map == kMapDiagLast) {
    // symmetric problems of one size: every problem's off-diagonal tiles,
    // then the diagonal ones, each XCD running its share of the second part
    // last
    const int T = probs[0].tiles_n, od = T * (T - 1) / 2, n1 = nprob * od;
    const int l = xcd_split_remap(blockIdx.x, n1, nprob * T);
    if (l < 0) return;
    if (l < n1) {
      pi = l / od;
      unrank_strict_upper(l - pi * od, T, ti, tj);
    } else {
      pi = (l - n1) / T;
      ti = tj = l - n1 - pi * T;
    }
  } else {
    // kMapXcd: contiguous ranges per XCD; kMapDeal (problems of different
    // sizes): chunks dealt over the XCDs; LIM: dispatch order
    const int t =
        LIM ? (int)blockIdx.x : (map == kMapDeal ? deal_chunks(blockIdx.x) : xcd_remap(blockIdx.x, gridDim.x));
    if (t >= total_tiles) return;
    pi = find_problem_gemm(probs, nprob, t);
    lt = t - probs[pi].tile_begin;
    const int tn = probs[pi].tiles_n;
    if (probs[pi].sym) unrank_upper(lt, tn, ti, tj);
    else if (!LIM) {
      // column-major over the output tiles: neighbouring workgroups (one XCD,
      // one L2) share the column block of B and walk the row blocks of A
      // (preconditioning Lr G: G's 128-column slab is fetched once per matrix)
      const int tm = (probs[pi].M + kTile - 1) / kTile;
      tj = lt / tm;
      ti = lt - tj * tm;
    } else {
      ti = lt / tn;
      tj = lt % tn;
    }
  }
  const GemmProblem P = probs[pi];
  const int m0 = ti * kTile, n0 = tj * TN;
  if (LIM && P.mcount && m0 >= *P.mcount) return;

  Operand<SA> A{reinterpret_cast<const SA*>(P.A), P.lda, P.a_rows, P.a_cols, P.a_aligned != 0};
  Operand<SB> B{reinterpret_cast<const SB*>(P.B), P.ldb, P.b_rows, P.b_cols, P.b_aligned != 0};
  int K = P.K;
  if (LIM && P.kcount) {
    const int cnt = *P.kcount;
    if (P.ksplit > 0) {
      const int kc = ((cnt + P.ksplit - 1) / P.ksplit + 15) & ~15;
      const int k0 = P.koff * kc;
      K = max(0, min(kc, cnt - k0));
      if (K > 0) {
        if (LA == kLayoutK) A.ptr += (int64_t)k0 * A.ld; else A.ptr += k0;
        if (LB == kLayoutK) B.ptr += (int64_t)k0 * B.ld; else B.ptr += k0;
        if (LA == kLayoutK) A.rows -= k0; else A.cols -= k0;
        if (LB == kLayoutK) B.rows -= k0; else B.cols -= k0;
      }
    } else {
      K = min(K, max(0, cnt - P.koff));
    }
    // the k-extent is the stored rows of a k-major operand, else its columns
    if (LA == kLayoutK) A.rows = min(A.rows, K); else A.cols = min(A.cols, K);
    if (LB == kLayoutK) B.rows = min(B.rows, K); else B.cols = min(B.cols, K);
  }
  WaveAcc<float, WN> acc;
  acc.zero();
  tile_mma<float, SA, LA, SB, LB, WN>(acc, A, B, m0, n0, K, sa0, sa1, sb0, sb1, P.sym && ti == tj);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const bool diag = P.sym && ti == tj;
  // the squares of wave_role: on a diagonal tile waves 1 and 2 share the
  // upper-right square (block rows of its top and bottom halves)
  const bool helper = diag && wave == 2;
  const int wm0 = m0 + (helper ? 0 : (wave >> 1) * kWaveTile),
            wn0 = n0 + (helper ? kWaveTile : (wave & 1) * kWaveTile * WN);
  typedef Mfma<float> F;
  if constexpr (!std::is_same<SGG, void>::value) {
    // plain outputs only (preconditioning); P.gD set: P with the fused graft
    // pass 1, else a plain store (the intermediate G Rr of two-sided blocks)
    const bool graft = P.gD != nullptr;
    {
      __shared__ double gred[kThreads / 64];
      float smg = 0.f, sps = 0.f;
      const bool vec = m0 + kTile <= P.M && n0 + TN <= P.N && (P.ldc & 3) == 0 && (P.ldg & 3) == 0 &&
                       (reinterpret_cast<uintptr_t>(P.C) & 15) == 0 && (reinterpret_cast<uintptr_t>(P.gD) & 15) == 0 &&
                       (reinterpret_cast<uintptr_t>(P.gG) & (4 * sizeof(SGG) - 1)) == 0;
      const bool rows16 = m0 + kTile <= P.M && n0 + TN <= P.N && (P.ldc & 3) == 0 &&
                          (reinterpret_cast<uintptr_t>(P.C) & 15) == 0;
      // a block row of the wave's accumulators (64 columns at a time) goes
      // through the wave's own LDS slice; the graft work then walks it row by
      // row (rolled loops, so the epilogue keeps the main loop's register
      // budget)
      float* epi = reinterpret_cast<float*>(wave == 0 ? sa0 : (wave == 1 ? sa1 : (wave == 2 ? sb0 : sb1)));
#pragma unroll
      for (int ih = 0; ih < WaveAcc<float>::NB * WN; ++ih) {
        const int i = ih / WN, h = ih % WN;
#pragma unroll
        for (int j = 0; j < WaveAcc<float>::NB; ++j)
#pragma unroll
          for (int v = 0; v < F::kAcc; ++v)
            epi[F::row(lane, v) * kWaveTile + j * F::kM + F::col(lane)] = P.alpha * acc.c[i][h * WaveAcc<float>::NB + j][v];
        const int r0 = wm0 + i * F::kM, c0 = wn0 + h * kWaveTile;
        if (!graft && rows16) {
          epi_rows(epi, P.C + (int64_t)r0 * P.ldc + c0, P.ldc, lane);
        } else if (!graft) {
#pragma unroll 1
          for (int idx = lane; idx < F::kM * kWaveTile; idx += 64) {
            const int r = r0 + idx / kWaveTile, c = c0 + idx % kWaveTile;
            if (r < P.M && c < P.N) gstore<float>(P.C + (int64_t)r * P.ldc + c, epi[idx]);
          }
        } else if (vec) {
          constexpr int kSeg = kWaveTile / 4;
#pragma unroll 1
          for (int k = 0; k < F::kM * kSeg / 64; ++k) {
            const int idx = lane + 64 * k, rr = idx / kSeg, c4 = (idx % kSeg) * 4;
            const f4v pv = *reinterpret_cast<const f4v*>(epi + rr * kWaveTile + c4);
            const int64_t gi = (int64_t)(r0 + rr) * P.ldg + c0 + c4;
            gstore<f4v>(P.C + (int64_t)(r0 + rr) * P.ldc + c0 + c4, pv);
            float g[4];
            G4<SGG>::load(P.gG, gi, g);
            f4v d = gload<f4v>(P.gD + gi);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              d[e] += g[e] * g[e];
              const float u = ada_dir(g[e], d[e]);
              smg += u * u;
              sps += pv[e] * pv[e];
            }
            gstore<f4v>(P.gD + gi, d);
          }
        } else {
#pragma unroll 1
          for (int idx = lane; idx < F::kM * kWaveTile; idx += 64) {
            const int rr = idx / kWaveTile, cc = idx % kWaveTile;
            const int r = r0 + rr, c = c0 + cc;
            if (r >= P.M || c >= P.N) continue;
            const float x = epi[rr * kWaveTile + cc];
            gstore<float>(P.C + (int64_t)r * P.ldc + c, x);
            const int64_t gi = (int64_t)r * P.ldg + c;
            const float g = load_g<SGG>(P.gG, gi);
            const float d = gload<float>(P.gD + gi) + g * g;
            gstore<float>(P.gD + gi, d);
            const float u = ada_dir(g, d);
            smg += u * u;
            sps += x * x;
          }
        }
      }
      if (graft) {
        const double a = block_sum((double)smg, gred);
        const double b = block_sum((double)sps, gred);
        if (threadIdx.x == 0) {
          P.gpart[2 * (P.part_base + lt) + 0] = a;
          P.gpart[2 * (P.part_base + lt) + 1] = b;
        }
      }
      return;
    }
  }
#if SHP_EPI_VEC
  // Symmetric output, off-diagonal full tile: mirrored values go out as
  // 16-byte stores (a lane's 4 consecutive rows are 4 consecutive columns of
  // the transposed tile).  The old output is symmetric too, so the four old
  // values of rows r..r+3, column c are one 16-byte load of row c (the
  // mirror this lane then overwrites; no other lane or workgroup touches it).
  if constexpr (WN == 1)
  if (P.sym && !diag && m0 + kTile <= P.M && n0 + kTile <= P.N && (P.ldc & 3) == 0 &&
      (reinterpret_cast<uintptr_t>(P.C) & 15) == 0) {
#pragma unroll
    for (int i = 0; i < WaveAcc<float>::NB; ++i)
#pragma unroll
      for (int j = 0; j < WaveAcc<float>::NB; ++j)
#pragma unroll
        for (int g = 0; g < F::kAcc / 4; ++g) {
          const int r = wm0 + i * F::kM + F::row(lane, 4 * g);
          const int c = wn0 + j * F::kM + F::col(lane);
          typedef float f4 __attribute__((ext_vector_type(4)));
          f4 w, old = {0.f, 0.f, 0.f, 0.f};
          if (P.beta != 0.f) old = gload<f4>(P.C + (int64_t)c * P.ldc + r);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float x = P.alpha * acc.c[i][j][4 * g + q];
            if (P.beta != 0.f) x += P.beta * old[q];
            gstore<float>(P.C + (int64_t)(r + q) * P.ldc + c, x);
            w[q] = x;
          }
          gstore<f4>(P.C + (int64_t)c * P.ldc + r, w);
        }
    return;
  }
  // Full tile of a plain output: rows through LDS, 16-byte row segments
  // (not compiled into the row x row instantiation, which only forms
  // symmetric statistics and would lose an occupancy step to it).
  if constexpr (!(LA == kLayoutRow && LB == kLayoutRow))
  if (!P.sym && m0 + kTile <= P.M && n0 + TN <= P.N && (P.ldc & 3) == 0 &&
      (reinterpret_cast<uintptr_t>(P.C) & 15) == 0) {
    float* epi = reinterpret_cast<float*>(wave == 0 ? sa0 : (wave == 1 ? sa1 : (wave == 2 ? sb0 : sb1)));
#pragma unroll
    for (int ih = 0; ih < WaveAcc<float>::NB * WN; ++ih) {
      const int i = ih / WN, h = ih % WN;
      const int c0 = wn0 + h * kWaveTile;
#pragma unroll
      for (int j = 0; j < WaveAcc<float>::NB; ++j)
#pragma unroll
        for (int v = 0; v < F::kAcc; ++v) {
          const int r = wm0 + i * F::kM + F::row(lane, v);
          const int c = c0 + j * F::kM + F::col(lane);
          float x = P.alpha * acc.c[i][h * WaveAcc<float>::NB + j][v];
          if (P.beta != 0.f) x += P.beta * gload<float>(P.C + (int64_t)r * P.ldc + c);
          epi[F::row(lane, v) * kWaveTile + j * F::kM + F::col(lane)] = x;
        }
      epi_rows(epi, P.C + (int64_t)(wm0 + i * F::kM) * P.ldc + c0, P.ldc, lane);
    }
    return;
  }
#endif
#pragma unroll
  for (int i = 0; i < WaveAcc<float>::NB; ++i)
#pragma unroll
    for (int j = 0; j < WaveAcc<float, WN>::NBJ; ++j)
#pragma unroll
      for (int v = 0; v < F::kAcc; ++v) {
        const int r = wm0 + i * F::kM + F::row(lane, v);
        const int c = wn0 + j * F::kM + F::col(lane);
        if (diag && wave == 1 && i >= WaveAcc<float>::NB / 2) continue;
        if (helper && i < WaveAcc<float>::NB / 2) continue;
        if (r >= P.M || c >= P.N) continue;
        if (diag && r > c) continue;
        float x = P.alpha * acc.c[i][j][v];
        if (P.beta != 0.f) x += P.beta * gload<float>(P.C + (int64_t)r * P.ldc + c);
        gstore<float>(P.C + (int64_t)r * P.ldc + c, x);
        if (P.sym && r != c) gstore<float>(P.C + (int64_t)c * P.ldc + r, x);
      }
}

// ============================================================================
// Coupled Newton iteration (Algorithm 1), grouped over matrices.
// ============================================================================
enum : int { kActive = -1 };
enum : int { kConverged = 0, kStagnated = 1, kMaxIter = 2, kDiverged = 3, kNotPD = 4 };
// warm phase only: the warm start was given up, the matrix takes the cold start
enum : int { kWarmAbort = 5 };

constexpr float kStagGate = 1e-3f;  // stagnation is tested only below this residual
constexpr float kDivergeAt = 1e6f;  // residual above this (or non-finite) diverged

// Per-matrix iteration state (device).
struct RootState {
  int status;        // kActive or a final code
  int iters;         // iterations of the current phase
  int parity;        // buffer index holding the current X and M
  int iters_fp32;    // iterations spent in the fp32 phase
  unsigned resid_bits;  // running max |M - I| of the iteration in flight (float bits)
  float resid;       // residual after the last iteration
  int escalate;      // AUTO policy: redo in fp64
  int precision;     // 32 or 64: phase that produced the result
  int sv_done;       // MaxSV stopped
  int sv_steps;      // MaxSV power steps taken
  int lz_done;       // Lanczos condition witness stopped (AUTO pre-escalation)
  int lz_steps;      // Lanczos steps taken
  double lz_beta;    // last off-diagonal of the Lanczos tridiagonal
  double lz_theta;   // its smallest Ritz value after the last step
  double z;          // scaling of M0 = z A_d: (1 + p) / (2 ||A_d||_F), times zc
  double zc;         // tightening factor of the power-bound scaling (1: Frobenius)
  double eps_eff;    // damping added
  double lam_max;    // MaxSV estimate (relative damping)
  double diag_min;   // smallest diagonal entry of A_d
  // warm start (coupled-Newton appendix)
  int warm;          // 0 not tried, 1 result from the warm iteration, 2 warm aborted (cold result)
  int warm_iters;    // iterations of the warm phase
  int grew;          // consecutive residual increases in the warm phase
  unsigned xmax_bits;  // max|X| of the new iterate (float bits)
  unsigned mmax_bits;  // max|M| of the new iterate
  unsigned comm_bits;  // max|XM - MX| of the new iterates
};

// Buffers of one matrix in one precision.
template <typename T>
struct NewtonJob {
  T* X[2];
  T* M[2];
  T* S[2];
  const float* A;   // input statistics (fp32, n x n)
  float* Xout;      // caller's output
  double* part;     // per-tile partial sums (tiles_n^2 x 2)
  double* vec;      // MaxSV vector and partials ((2 tiles_n + 1) n)
  int n;
  int tiles_n;      // ceil(n / 128)
  int up_begin;     // first logical upper-triangular tile
  int full_begin;   // first logical full-grid tile
  int flat_begin;   // first flat chunk (kFlatChunk elements)
};

// Elementwise passes that need no transpose walk each matrix as one
// contiguous array: a workgroup takes kFlatChunk consecutive elements of one
// job (16-byte vectors when n % 4 == 0, which keeps every vector inside one
// row).  A standalone copy of 96 matrices of 1024^2 streamed 6.2 TB/s this
// way against 5.05 over 128 x 128 tiles (128 separate 512-byte row segments
// per workgroup); in the library the output copy went from 144 to 134 us,
// the first-iteration pass (three in, three out) stayed at about 465 us.
constexpr int kFlatChunk = 4096;

template <typename T>
__device__ __forceinline__ int find_job_up(const NewtonJob<T>* jobs, int njobs, int t) {
  int lo = 0, hi = njobs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (jobs[mid].up_begin <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

template <typename T>
__device__ __forceinline__ int find_job_flat(const NewtonJob<T>* jobs, int njobs, int t) {
  int lo = 0, hi = njobs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (jobs[mid].flat_begin <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

template <typename T>
__device__ __forceinline__ int find_job_full(const NewtonJob<T>* jobs, int njobs, int t) {
  int lo = 0, hi = njobs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (jobs[mid].full_begin <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// One launch of a Newton iteration runs up to three independent products
// over all upper tiles of every active matrix.  Each product is
//   C[dst] = ca (B[a] B[b]) + cb B[e] + cg I      (+ max|C - I| when resid)
// over the six iterate buffers of a matrix, named by id:
//   0 X (current), 1 X (next), 2 M (current), 3 M (next), 4 S0, 5 S1.
// M1 = a I + b M (a = (p+1)/p, b = -1/p) is never stored: products with it
// are expanded into a plain product of stored buffers and the affine terms
// (X M1 = b X M + a X, M1 M = b M M + a M, M1 M1 = b^2 M M + 2ab M + a^2 I).
// Every factor is a polynomial in the same symmetric A, so every product is
// symmetric and only upper tiles are computed.
enum : int { kBufXc = 0, kBufXn = 1, kBufMc = 2, kBufMn = 3, kBufS0 = 4, kBufS1 = 5, kBufNone = -1 };

// amax (full products of the warm start only): max|C| into the matrix's
// monitor slot 1 xmax, 2 mmax or 3 comm.
enum : int { kAmaxNone = 0, kAmaxX = 1, kAmaxM = 2, kAmaxComm = 3 };

struct NewtonProd {
  int a, b, e, dst;  // buffer ids (e = kBufNone: no affine E term; dst = kBufNone: not stored)
  int resid, amax;
  double ca, cb, cg;
};

struct NewtonStage {
  int nprod, pad;
  NewtonProd q[3];
};

template <typename V>
__device__ __forceinline__ V pick3(int i, V x0, V x1, V x2) {
  return i == 0 ? x0 : (i == 1 ? x1 : x2);
}

template <typename T>
__device__ __forceinline__ T* newton_buf(const NewtonJob<T>* J, int par, int id) {
  // the table is read with run-time indices (a local copy of the struct would
  // be placed in scratch)
  if (id < 2) return J->X[(id & 1) ^ par];
  if (id < 4) return J->M[(id & 1) ^ par];
  return J->S[id & 1];
}

// Upper tile t of a product launch, packed as job << 10 | ti << 5 | tj
// (tile indices < 32: n <= 4096), so a workgroup finds its tile with one load.
__host__ __device__ __forceinline__ uint32_t pack_tile(int j, int ti, int tj) {
  return ((uint32_t)j << 10) | ((uint32_t)ti << 5) | (uint32_t)tj;
}

// Compact list of the tiles of the matrices still active, in two parts:
// tlist[0, tcount[1]) the early tiles, then tlist[tcount[1], tcount[0]) the
// late ones, each part in job order.  tmap holds every tile of a launch
// (job-major: the upper tiles of the symmetric products, row-major, or the
// full grid of the warm start's) and ubegin[j] the first of job j
// (ubegin[njobs] = their number).  diag_last (upper tiles only): the
// diagonal tiles, which cost less than the others, form the late part, and
// the launch runs each XCD's share of them last; else every tile is early.
// A job's upper tiles end with its last diagonal tile (T-1, T-1), so it has
// that tile's row + 1 of them.  Called by one whole workgroup; st must be
// final for every job (the caller's threads have passed a barrier since they
// last wrote it).
__device__ __forceinline__ void build_tile_list(const RootState* __restrict__ st, int njobs,
                                                const uint32_t* __restrict__ tmap, const int* __restrict__ ubegin,
                                                int diag_last, uint32_t* __restrict__ tlist,
                                                int* __restrict__ tcount) {
  __shared__ int scan[2][kThreads];
  __shared__ int base[2];
  __shared__ int red[2][kThreads / 64];
  auto ndiag = [&](int j) { return (int)((tmap[ubegin[j + 1] - 1] >> 5) & 31) + 1; };
  // tiles of the active matrices and their late ones: where the late part starts
  int all = 0, late = 0;
  for (int j = threadIdx.x; j < njobs; j += kThreads)
    if (st[j].status == kActive) {
      all += ubegin[j + 1] - ubegin[j];
      if (diag_last) late += ndiag(j);
    }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    all += __shfl_xor(all, o, 64);
    late += __shfl_xor(late, o, 64);
  }
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = all;
    red[1][threadIdx.x >> 6] = late;
  }
  if (threadIdx.x == 0) base[0] = base[1] = 0;
  __syncthreads();
  int early = 0;
  for (int w = 0; w < kThreads / 64; ++w) early += red[0][w] - red[1][w];
  for (int j0 = 0; j0 < njobs; j0 += kThreads) {
    const int j = j0 + (int)threadIdx.x;
    const bool on = j < njobs && st[j].status == kActive;
    const bool mv = on && diag_last;
    const int b = on ? ubegin[j] : 0, n = on ? ubegin[j + 1] - b : 0;
    const int n1 = mv ? ndiag(j) : 0, n0 = n - n1;
    scan[0][threadIdx.x] = n0;
    scan[1][threadIdx.x] = n1;
    __syncthreads();
    for (int o = 1; o < kThreads; o <<= 1) {  // inclusive scans
      const int v0 = (int)threadIdx.x >= o ? scan[0][threadIdx.x - o] : 0;
      const int v1 = (int)threadIdx.x >= o ? scan[1][threadIdx.x - o] : 0;
      __syncthreads();
      scan[0][threadIdx.x] += v0;
      scan[1][threadIdx.x] += v1;
      __syncthreads();
    }
    int o0 = base[0] + scan[0][threadIdx.x] - n0;
    int o1 = early + base[1] + scan[1][threadIdx.x] - n1;
    if (mv) {
      for (int k = 0; k < n; ++k) {
        const uint32_t c = tmap[b + k];
        if (((c >> 5) & 31) == (c & 31)) tlist[o1++] = c;
        else tlist[o0++] = c;
      }
    } else {
      for (int k = 0; k < n; ++k) tlist[o0 + k] = tmap[b + k];
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      base[0] += scan[0][kThreads - 1];
      base[1] += scan[1][kThreads - 1];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    tcount[0] = early + base[1];
    tcount[1] = early;
  }
}

__global__ __launch_bounds__(kThreads) void tile_list_kernel(const RootState* __restrict__ st, int njobs,
                                                            const uint32_t* __restrict__ tmap,
                                                            const int* __restrict__ ubegin, int diag_last,
                                                            uint32_t* __restrict__ tlist, int* __restrict__ tcount) {
  build_tile_list(st, njobs, tmap, ubegin, diag_last, tlist, tcount);
}

// tlist / tcount: the compact upper-tile list of the matrices still active
// (build_tile_list: early tiles, then any late diagonal ones); the grid is
// sized for every upper tile (plus the slack of xcd_split_remap), and the
// workgroups past the work return at once.  The workgroup -> tile remap is
// taken over the active part only, so the work of a few remaining matrices
// still spreads over every XCD.  Each XCD runs its share of the early tiles
// before its share of the late, cheaper diagonal ones (of the matrices of
// its own range), which evens out when its compute units finish.
template <typename T>
__global__ __launch_bounds__(kThreads, MinWaves<T>::value) void newton_stage_kernel(const NewtonJob<T>* __restrict__ jobs,
                                                               const uint32_t* __restrict__ tlist,
                                                               const int* __restrict__ tcount, int njobs,
                                                               RootState* __restrict__ st, NewtonStage S,
                                                               int mixed) {
  __shared__ __attribute__((aligned(16))) T sa0[StageElems<T, kLayoutK>::value], sa1[StageElems<T, kLayoutK>::value];
  __shared__ __attribute__((aligned(16))) T sb0[StageElems<T, kLayoutK>::value], sb1[StageElems<T, kLayoutK>::value];
  const int np = S.nprod;
  const int nt = tcount[0], ne = tcount[1];
  int l;
  if (mixed) {  // matrices of different sizes: chunks dealt over the XCDs
    l = deal_chunks(blockIdx.x);
    if (l >= np * nt) return;
  } else {
    l = xcd_split_remap(blockIdx.x, np * ne, np * (nt - ne));
    if (l < 0) return;
  }
  // the products of one tile run in neighbouring workgroups (shared operands)
  const int t = l / np, prod = l - t * np;
  const uint32_t code = tlist[t];
  const int j = (int)(code >> 10), ti = (int)((code >> 5) & 31), tj = (int)(code & 31);
  if (st[j].status != kActive) return;
  const NewtonJob<T>* J = jobs + j;
  const int par = st[j].parity;
  const int n = J->n;
  const int m0 = ti * kTile, n0 = tj * kTile;

  const int ia = pick3(prod, S.q[0].a, S.q[1].a, S.q[2].a);
  const int ib = pick3(prod, S.q[0].b, S.q[1].b, S.q[2].b);
  const int ie = pick3(prod, S.q[0].e, S.q[1].e, S.q[2].e);
  const int id = pick3(prod, S.q[0].dst, S.q[1].dst, S.q[2].dst);
  const bool resid = pick3(prod, S.q[0].resid, S.q[1].resid, S.q[2].resid) != 0;
  const T ca = (T)pick3(prod, S.q[0].ca, S.q[1].ca, S.q[2].ca);  // alpha, beta, gamma
  const T cb = (T)pick3(prod, S.q[0].cb, S.q[1].cb, S.q[2].cb);
  const T cg = (T)pick3(prod, S.q[0].cg, S.q[1].cg, S.q[2].cg);
  const T* pa = newton_buf(J, par, ia);
  const T* pb = newton_buf(J, par, ib);
  T* pc = newton_buf(J, par, id);
  const T* pe = ie >= 0 ? newton_buf(J, par, ie) : nullptr;  // E of the affine epilogue
  const bool al = (reinterpret_cast<uintptr_t>(pa) & 15) == 0 && (reinterpret_cast<uintptr_t>(pb) & 15) == 0 &&
                  ((n * (int)sizeof(T)) & 15) == 0;
  Operand<T> A{pa, n, n, n, al};
  Operand<T> B{pb, n, n, n, al};

  WaveAcc<T> acc;
  acc.zero();
  // All operands are symmetric, so both are read k-major (storage row = k).
  tile_mma<T, T, kLayoutK, T, kLayoutK>(acc, A, B, m0, n0, n, sa0, sa1, sb0, sb1, ti == tj);
  // value of output element (r, c) from its accumulator
  auto fin = [&](T v, int r, int c) -> T {
    T x = ca * v;
    if (pe) x += cb * gload<T>(pe + (int64_t)r * n + c);
    if (r == c) x += cg;
    return x;
  };

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const bool diag = ti == tj;
  // the squares of wave_role (waves 1 and 2 share the upper-right square of
  // a diagonal tile)
  const bool helper = diag && wave == 2;
  const int wm0 = m0 + (helper ? 0 : (wave >> 1) * kWaveTile), wn0 = n0 + (helper ? kWaveTile : (wave & 1) * kWaveTile);
  typedef Mfma<T> F;
  float rmax = 0.f;
  auto track = [&](T x, int r, int c) {
    if (resid) {
      float d = (float)fabs((double)x - (r == c ? 1.0 : 0.0));
      if (!(d <= 3.0e38f)) d = INFINITY;  // NaN or overflow
      rmax = rmax > d ? rmax : d;
    }
  };
#if SHP_EPI_VEC
  // Off-diagonal full tile of an fp32 product: the 4 consecutive rows a lane
  // holds (v = 4g .. 4g+3) are 4 consecutive columns of the mirrored tile,
  // written as one 16-byte store.
  if (sizeof(T) == 4 && !diag && m0 + kTile <= n && n0 + kTile <= n && (n & 3) == 0) {
#pragma unroll
    for (int i = 0; i < WaveAcc<T>::NB; ++i)
#pragma unroll
      for (int jj = 0; jj < WaveAcc<T>::NB; ++jj)
#pragma unroll
        for (int g = 0; g < F::kAcc / 4; ++g) {
          const int r = wm0 + i * F::kM + F::row(lane, 4 * g);
          const int c = wn0 + jj * F::kM + F::col(lane);
          typedef float f4 __attribute__((ext_vector_type(4)));
          f4 w;
          // E is exactly symmetric (iterates are stored mirrored), so the
          // four E values of rows r..r+3, column c are one 16-byte load of
          // row c: E[c][r..r+3].
          f4 e4 = {0.f, 0.f, 0.f, 0.f};
          if (pe) e4 = gload<f4>(reinterpret_cast<const float*>(pe) + (int64_t)c * n + r);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            T x = ca * acc.c[i][jj][4 * g + q] + cb * (T)e4[q];
            if (r + q == c) x += cg;
            w[q] = (float)x;
            gstore<T>(pc + (int64_t)(r + q) * n + c, x);
            track(x, r + q, c);
          }
          gstore<f4>(reinterpret_cast<float*>(pc) + (int64_t)c * n + r, w);
        }
  } else
#endif
  {
#pragma unroll
    for (int i = 0; i < WaveAcc<T>::NB; ++i)
#pragma unroll
      for (int jj = 0; jj < WaveAcc<T>::NB; ++jj)
#pragma unroll
        for (int v = 0; v < F::kAcc; ++v) {
          const int r = wm0 + i * F::kM + F::row(lane, v);
          const int c = wn0 + jj * F::kM + F::col(lane);
          if (diag && wave == 1 && i >= WaveAcc<T>::NB / 2) continue;
          if (helper && i < WaveAcc<T>::NB / 2) continue;
          if (r >= n || c >= n) continue;
          if (diag && r > c) continue;
          const T x = fin(acc.c[i][jj][v], r, c);
          gstore<T>(pc + (int64_t)r * n + c, x);
          if (r != c) gstore<T>(pc + (int64_t)c * n + r, x);
          track(x, r, c);
        }
  }
  if (resid) {
    rmax = wave_max(rmax);
    if (lane == 0 && rmax > 0.f) atomicMax(&st[j].resid_bits, __float_as_uint(rmax));
  }
}

// Warm start (coupled-Newton appendix: X0 = the previous root,
// M0 = X0^p A_d).  X0 does not commute with the new statistics, so neither X
// nor M stays symmetric: every product of the warm phase is a full n x n
// product of general matrices, over the full tile grid of every active
// matrix, with the program format of newton_stage_kernel:
//   C[dst] = ca (B[a] B[b]) + cb B[e] + cg I
// The left operand is staged in the row layout (its contraction index is
// the storage column), the right one k-major.  dst == kBufNone stores
// nothing (the commutator only needs its largest entry); q.amax adds max|C|
// to a monitor slot, q.resid max|C - I| to the residual.
// tlist / tcount / mixed: as newton_stage_kernel, over the full tile grid.
template <typename T>
__global__ __launch_bounds__(kThreads, kMinWaves) void newton_dense_kernel(const NewtonJob<T>* __restrict__ jobs,
                                                                          const uint32_t* __restrict__ tlist,
                                                                          const int* __restrict__ tcount,
                                                                          int njobs, RootState* __restrict__ st,
                                                                          NewtonStage S, int mixed) {
  __shared__ __attribute__((aligned(16))) T sa0[StageElems<T, kLayoutRow>::value], sa1[StageElems<T, kLayoutRow>::value];
  __shared__ __attribute__((aligned(16))) T sb0[StageElems<T, kLayoutK>::value], sb1[StageElems<T, kLayoutK>::value];
  const int np = S.nprod;
  const int nwork = np * *tcount;
  int l;
  if (mixed) {
    l = deal_chunks(blockIdx.x);
    if (l >= nwork) return;
  } else {
    if ((int)blockIdx.x >= nwork) return;
    l = xcd_remap(blockIdx.x, nwork);
  }
  const int t = l / np, prod = l - t * np;
  const uint32_t code = tlist[t];
  const int j = (int)(code >> 10), ti = (int)((code >> 5) & 31), tj = (int)(code & 31);
  if (j >= njobs || st[j].status != kActive) return;
  const NewtonJob<T>* J = jobs + j;
  const int par = st[j].parity;
  const int n = J->n;
  const int m0 = ti * kTile, n0 = tj * kTile;

  const int ia = pick3(prod, S.q[0].a, S.q[1].a, S.q[2].a);
  const int ib = pick3(prod, S.q[0].b, S.q[1].b, S.q[2].b);
  const int ie = pick3(prod, S.q[0].e, S.q[1].e, S.q[2].e);
  const int id = pick3(prod, S.q[0].dst, S.q[1].dst, S.q[2].dst);
  const bool resid = pick3(prod, S.q[0].resid, S.q[1].resid, S.q[2].resid) != 0;
  const int amax = pick3(prod, S.q[0].amax, S.q[1].amax, S.q[2].amax);
  const T ca = (T)pick3(prod, S.q[0].ca, S.q[1].ca, S.q[2].ca);
  const T cb = (T)pick3(prod, S.q[0].cb, S.q[1].cb, S.q[2].cb);
  const T cg = (T)pick3(prod, S.q[0].cg, S.q[1].cg, S.q[2].cg);
  const T* pa = newton_buf(J, par, ia);
  const T* pb = newton_buf(J, par, ib);
  T* pc = id >= 0 ? newton_buf(J, par, id) : nullptr;
  const T* pe = ie >= 0 ? newton_buf(J, par, ie) : nullptr;
  const bool al = (reinterpret_cast<uintptr_t>(pa) & 15) == 0 && (reinterpret_cast<uintptr_t>(pb) & 15) == 0 &&
                  ((n * (int)sizeof(T)) & 15) == 0;
  Operand<T> A{pa, n, n, n, al};
  Operand<T> B{pb, n, n, n, al};

  WaveAcc<T> acc;
  acc.zero();
  tile_mma<T, T, kLayoutRow, T, kLayoutK>(acc, A, B, m0, n0, n, sa0, sa1, sb0, sb1);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm0 = m0 + (wave >> 1) * kWaveTile, wn0 = n0 + (wave & 1) * kWaveTile;
  typedef Mfma<T> F;
  float rmax = 0.f, cmax = 0.f;
#pragma unroll
  for (int i = 0; i < WaveAcc<T>::NB; ++i)
#pragma unroll
    for (int jj = 0; jj < WaveAcc<T>::NB; ++jj)
#pragma unroll
      for (int v = 0; v < F::kAcc; ++v) {
        const int r = wm0 + i * F::kM + F::row(lane, v);
        const int c = wn0 + jj * F::kM + F::col(lane);
        if (r >= n || c >= n) continue;
        T x = ca * acc.c[i][jj][v];
        if (pe) x += cb * pe[(int64_t)r * n + c];
        if (r == c) x += cg;
        if (pc) gstore<T>(pc + (int64_t)r * n + c, x);
        if (resid) {
          float d = (float)fabs((double)x - (r == c ? 1.0 : 0.0));
          if (!(d <= 3.0e38f)) d = INFINITY;  // NaN or overflow
          rmax = rmax > d ? rmax : d;
        }
        if (amax) {
          float d = (float)fabs((double)x);
          if (!(d <= 3.0e38f)) d = INFINITY;
          cmax = cmax > d ? cmax : d;
        }
      }
  if (resid) {
    rmax = wave_max(rmax);
    if (lane == 0 && rmax > 0.f) atomicMax(&st[j].resid_bits, __float_as_uint(rmax));
  }
  if (amax) {
    cmax = wave_max(cmax);
    unsigned* slot = amax == kAmaxX ? &st[j].xmax_bits : (amax == kAmaxM ? &st[j].mmax_bits : &st[j].comm_bits);
    if (lane == 0 && cmax > 0.f) atomicMax(slot, __float_as_uint(cmax));
  }
}

// Warm start, set-up pass over the full tile grid: A_d = A_s + eps_eff I
// into the next-M buffer (the right factor of M0 = X0^p A_d); in fp64 the
// caller's X0 (fp32) is also copied into the current-X buffer (in fp32 that
// buffer is the caller's X itself).
template <typename T>
__global__ __launch_bounds__(kThreads) void warm_init_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs,
                                                            const RootState* __restrict__ st, int total_full) {
  __shared__ float lds[kTile * 33];
  const int t = blockIdx.x;
  if (t >= total_full) return;
  const int j = find_job_full(jobs, njobs, t);
  if (st[j].status != kActive) return;
  const NewtonJob<T> J = jobs[j];
  const int lt = t - J.full_begin;
  const int ti = lt / J.tiles_n, tj = lt % J.tiles_n;
  const double e = st[j].eps_eff;
  const int n = J.n;
  T* Ad = J.M[1];
  sym_tile_pass(J.A, n, ti, tj, lds, [&](int r, int c, double s) {
    Ad[(int64_t)r * n + c] = (T)(s + (r == c ? e : 0.0));
  });
  if (sizeof(T) == 8) {
    const int r0 = ti * kTile, c0 = tj * kTile;
    for (int q = threadIdx.x; q < kTile * kTile; q += kThreads) {
      const int r = r0 + (q >> 7), c = c0 + (q & 127);
      if (r < n && c < n) J.X[0][(int64_t)r * n + c] = (T)J.Xout[(int64_t)r * n + c];
    }
  }
}

// Warm-phase state machine, one workgroup (rules of the oracle's warm
// iteration: Algorithm 1's stop test, R3's floor and divergence limits, and
// the commutator monitor of the coupled-Newton appendix).  count[0]:
// matrices still in the warm phase; count[1]: matrices whose warm start was
// given up.
//   init != 0: residual of M0 = X0^p A_d only.
__global__ __launch_bounds__(kThreads) void root_warm_update_kernel(RootState* __restrict__ st, int njobs, int init,
                                                                   float tol, float comm_tol, int max_iters,
                                                                   int* __restrict__ count,
                                                                   const uint32_t* __restrict__ tmap,
                                                                   const int* __restrict__ ubegin,
                                                                   uint32_t* __restrict__ tlist,
                                                                   int* __restrict__ tcount) {
  __shared__ int red[2 * (kThreads / 64)];
  int active = 0, aborted = 0;
  for (int j = threadIdx.x; j < njobs; j += kThreads) {
    RootState& s = st[j];
    if (s.status != kActive) {
      aborted += s.status == kWarmAbort;
      continue;
    }
    const float r = __uint_as_float(s.resid_bits);
    s.resid_bits = 0u;
    bool abort = false;
    if (init) {
      s.resid = r;
      if (r <= tol) s.status = kConverged;
      else if (!(r <= kDivergeAt) || max_iters < 1) abort = true;
    } else {
      s.parity ^= 1;
      s.iters += 1;
      const float prev = s.resid;
      s.resid = r;
      const float c = __uint_as_float(s.comm_bits);
      const float scale = __uint_as_float(s.xmax_bits) * __uint_as_float(s.mmax_bits);
      s.comm_bits = s.xmax_bits = s.mmax_bits = 0u;
      s.grew = r > prev ? s.grew + 1 : 0;
      if (!(c <= comm_tol * scale) || s.grew >= 2) abort = true;
      else if (r <= tol) s.status = kConverged;
      else if (prev < kStagGate && r >= prev) s.status = kStagnated;
      else if (!(r <= kDivergeAt) || s.iters >= max_iters) abort = true;
    }
    if (abort) s.status = kWarmAbort;
    if (s.status == kActive) ++active;
    else aborted += s.status == kWarmAbort;
  }
  int a = active, f = aborted;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    a += __shfl_xor(a, o, 64);
    f += __shfl_xor(f, o, 64);
  }
  if ((threadIdx.x & 63) == 0) {
    red[threadIdx.x >> 6] = a;
    red[kThreads / 64 + (threadIdx.x >> 6)] = f;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int sa = 0, sf = 0;
    for (int w = 0; w < kThreads / 64; ++w) {
      sa += red[w];
      sf += red[kThreads / 64 + w];
    }
    count[0] = sa;
    count[1] = sf;
  }
  // the next iteration's tiles (full grid) of the matrices still in the phase
  build_tile_list(st, njobs, tmap, ubegin, 0, tlist, tcount);
}

// End of the warm phase: records its outcome (warm_out, device int32
// [njobs][2] = {outcome, warm iterations}, may be NULL) and hands the
// matrices whose warm start was given up to the cold start.
__global__ void root_warm_finish_kernel(RootState* __restrict__ st, int njobs, int32_t* __restrict__ warm_out) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= njobs) return;
  RootState& s = st[j];
  if (s.status == kNotPD) {
    s.warm = 0;
    s.warm_iters = 0;
  } else if (s.status == kWarmAbort) {
    s.warm = 2;
    s.warm_iters = s.iters;
    s.status = kActive;
    s.iters = 0;
    s.parity = 0;
    s.resid_bits = 0u;
    s.resid = INFINITY;
    s.grew = 0;
  } else {
    s.warm = 1;
    s.warm_iters = s.iters;
  }
  if (warm_out) {
    warm_out[2 * j] = s.warm;
    warm_out[2 * j + 1] = s.warm_iters;
  }
}

// ---------------------------------------------------------------------------
// Prologue.  MaxSV (Algorithm 1): power iteration on A_s = (A + A^T)/2 in
// fp64 arithmetic, one workgroup per matrix, v0 = ones, Rayleigh quotient,
// relative stop.
// ---------------------------------------------------------------------------
// MaxSV, one power step over all matrices, in two launches.  Tile pass:
// workgroup (matrix, ti, tj) stages tile A[ti, tj] in LDS and writes its
// row partials (A vh)_rows and column partials (A^T vh)_cols.  Reduce pass
// (maxsv_reduce_kernel): the partials in a fixed order give
// v = A_s vh = (A vh + A^T vh) / 2, the Rayleigh quotient lambda = vh . v,
// the stop test |lambda - lambda_old| <= tol lambda, and the next
// vh = v / |v|.  No workgroup waits on or signals another (a device-scope
// fence per workgroup would write back and invalidate the XCD L2s).
// Vector layout per matrix (doubles): [0, n) vh, [n, n + T n) row partials
// by tile column, [n + T n, n + 2 T n) column partials by tile row.
// lanczos: the same pass for a Lanczos step (lanczos_reduce_kernel), gated
// by that iteration's own stop flag.
template <typename T>
__global__ __launch_bounds__(kThreads) void maxsv_step_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs,
                                                             const RootState* __restrict__ st, int total_full,
                                                             int lanczos) {
  // the tile is staged in two halves of 64 rows (33 KB of LDS, so four
  // workgroups share a CU and hide each other's loads)
  constexpr int kHalf = kTile / 2;
  __shared__ float tile[kHalf * (kTile + 1)];
  __shared__ double vr[kTile], vc[kTile];       // v on the tile's rows and columns
  __shared__ double rsum[4][kHalf];             // row partials of a half, by column quarter
  __shared__ double csum[2][kTile];             // column partials, by row half of a half
  const int t = blockIdx.x;
  if (t >= total_full) return;
  const int j = find_job_full(jobs, njobs, t);
  if (st[j].status != kActive || (lanczos ? st[j].lz_done : st[j].sv_done)) return;
  const NewtonJob<T>* J = jobs + j;
  const int n = J->n, TN = J->tiles_n;
  const int lt = t - J->full_begin;
  const int ti = lt / TN, tj = lt % TN;
  const int r0 = ti * kTile, c0 = tj * kTile;
  double* vh = J->vec;
  double* prow = J->vec + n;
  double* pcol = J->vec + n + (int64_t)TN * n;
  const float* A = J->A;
  if (threadIdx.x < kTile) {
    const int i = threadIdx.x;
    vc[i] = c0 + i < n ? vh[c0 + i] : 0.0;
    vr[i] = r0 + i < n ? vh[r0 + i] : 0.0;
  }
  const bool vec = (n & 3) == 0 && r0 + kTile <= n && c0 + kTile <= n && (reinterpret_cast<uintptr_t>(A) & 15) == 0;
  const int rq = threadIdx.x & (kHalf - 1), quarter = threadIdx.x >> 6;  // row dots: 4 column quarters
  const int cq = threadIdx.x & (kTile - 1), rh = threadIdx.x >> 7;       // column dots: 2 row halves
  double cacc = 0.0;
  for (int h = 0; h < 2; ++h) {
    const int hr0 = r0 + h * kHalf;
    __syncthreads();  // the previous half's tile has been read
    if (vec) {
      for (int e = threadIdx.x; e < kHalf * kTile / 4; e += kThreads) {
        const int r = e >> 5, c = (e & 31) * 4;
        const f4v v = gload<f4v>(A + (int64_t)(hr0 + r) * n + c0 + c);
        float* d = tile + r * (kTile + 1) + c;
        d[0] = v[0]; d[1] = v[1]; d[2] = v[2]; d[3] = v[3];
      }
    } else {
      for (int e = threadIdx.x; e < kHalf * kTile; e += kThreads) {
        const int r = e >> 7, c = e & 127;
        tile[r * (kTile + 1) + c] = (hr0 + r < n && c0 + c < n) ? A[(int64_t)(hr0 + r) * n + c0 + c] : 0.f;
      }
    }
    __syncthreads();
    // (A v) on the half's rows, each dot product over four column quarters
    double racc = 0.0;
#pragma unroll 8
    for (int c = quarter * 32; c < quarter * 32 + 32; ++c) racc += (double)tile[rq * (kTile + 1) + c] * vc[c];
    rsum[quarter][rq] = racc;
    // (A^T v) on the tile's columns, accumulated over both halves
#pragma unroll 8
    for (int r = rh * 32; r < rh * 32 + 32; ++r) cacc += (double)tile[r * (kTile + 1) + cq] * vr[h * kHalf + r];
    __syncthreads();
    if (threadIdx.x < kHalf && hr0 + threadIdx.x < n)
      prow[(int64_t)tj * n + hr0 + threadIdx.x] =
          rsum[0][threadIdx.x] + rsum[1][threadIdx.x] + rsum[2][threadIdx.x] + rsum[3][threadIdx.x];
  }
  csum[rh][cq] = cacc;
  __syncthreads();
  if (threadIdx.x < kTile && c0 + threadIdx.x < n)
    pcol[(int64_t)ti * n + c0 + threadIdx.x] = csum[0][threadIdx.x] + csum[1][threadIdx.x];
}

// MaxSV reduction, one workgroup per matrix: v = (A v + A^T v) / 2 from the
// tile partials (fixed order), lambda = vh . v, vh = v / ||v||.  The kernel
// boundary after the tile pass makes every partial visible.
constexpr int kSvThreads = 1024;  // threads of the MaxSV reduction (one workgroup per matrix)

__device__ __forceinline__ double sv_block_sum(double v, double* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int w = 0; w < kSvThreads / 64; ++w) s += red[w];
  return s;
}

template <typename T>
__global__ __launch_bounds__(kSvThreads) void maxsv_reduce_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs,
                                                                 RootState* __restrict__ st, double tol, double eps,
                                                                 int last_step) {
  __shared__ double red[kSvThreads / 64];
  const int j = blockIdx.x;
  if (j >= njobs || st[j].status != kActive || st[j].sv_done) return;
  const NewtonJob<T>* J = jobs + j;
  const int n = J->n, TN = J->tiles_n;
  double* vh = J->vec;
  double* prow = J->vec + n;
  double* pcol = J->vec + n + (int64_t)TN * n;
  double q = 0.0, s2 = 0.0;
  for (int i = threadIdx.x; i < n; i += kSvThreads) {
    double a = 0.0, b = 0.0;
    for (int k = 0; k < TN; ++k) {
      a += prow[(int64_t)k * n + i];
      b += pcol[(int64_t)k * n + i];
    }
    const double v = 0.5 * (a + b);
    q += vh[i] * v;
    s2 += v * v;
    prow[i] = v;  // row partials of tile column 0 are consumed: reuse as v
  }
  const double lam = sv_block_sum(q, red);
  const double nrm = sqrt(sv_block_sum(s2, red));
  const double lam_old = st[j].lam_max;
  for (int i = threadIdx.x; i < n; i += kSvThreads) vh[i] = nrm > 0.0 ? prow[i] / nrm : 0.0;
  if (threadIdx.x == 0) {
    st[j].lam_max = lam;
    st[j].eps_eff = eps * lam;
    st[j].sv_steps += 1;
    if (fabs(lam - lam_old) <= tol * fabs(lam) || last_step) st[j].sv_done = 1;
  }
}

// Starting vector of MaxSV: vh = ones / sqrt(n).
template <typename T>
__global__ void maxsv_init_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs, RootState* __restrict__ st) {
  const int j = blockIdx.x;
  if (j >= njobs) return;
  const int n = jobs[j].n;
  for (int i = threadIdx.x; i < n; i += blockDim.x) jobs[j].vec[i] = 1.0 / sqrt((double)n);
  if (threadIdx.x == 0) {
    st[j].lam_max = 0.0;
    st[j].sv_done = 0;
    st[j].sv_steps = 0;
  }
}

// ---------------------------------------------------------------------------
// AUTO pre-escalation: a Lanczos witness of the condition number.  k steps
// of the Lanczos iteration on A_d = A_s + eps_eff I (fp64 arithmetic, start
// ones / sqrt(n)) give a k x k tridiagonal T whose Ritz values lie inside
// [lambda_min(A_d), lambda_max(A_d)]; with the MaxSV Rayleigh quotient
// lambda_hat + eps_eff <= lambda_max(A_d),
//   kappa(A_d) >= kappa_lb = (lambda_hat + eps_eff) / theta_min(T).
// After the cold start the smallest scaled eigenvalue is at most
// (p + 1) / (2 kappa), so once (p + 1) / (2 kappa_lb) < m1, the smallest
// scaled eigenvalue that still converges within the fp32 cap, the fp32 phase
// is certain to end unaccepted for this matrix: it goes straight to fp64
// (status MAXITER, 0 fp32 iterations).  A matrix stops when that is shown,
// when theta_min has settled (relative change below 1e-2), when the Krylov
// space is exhausted, or after kmax steps; it then takes the fp32 phase as
// before.  Vector layout after MaxSV's: [n + 2 T n, 2 n + 2 T n) the previous
// Lanczos vector, then alpha[kLanczosMax], beta[kLanczosMax].
// ---------------------------------------------------------------------------
constexpr int kLanczosMax = 96;

template <typename T>
__global__ void lanczos_init_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs, RootState* __restrict__ st) {
  const int j = blockIdx.x;
  if (j >= njobs) return;
  const int n = jobs[j].n, TN = jobs[j].tiles_n;
  double* v = jobs[j].vec;
  double* vp = jobs[j].vec + n + 2 * (int64_t)TN * n;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    v[i] = 1.0 / sqrt((double)n);
    vp[i] = 0.0;
  }
  if (threadIdx.x == 0) {
    st[j].lz_done = st[j].status != kActive;
    st[j].lz_steps = 0;
    st[j].lz_beta = 0.0;
    st[j].lz_theta = INFINITY;
  }
}

// Number of eigenvalues of the symmetric tridiagonal (a[0..m), b[0..m-1))
// below x: negative pivots of the LDL^T factorisation of T - x I (Sturm).
__device__ inline int sturm_below(const double* a, const double* b, int m, double x) {
  int c = 0;
  double d = 1.0;
  for (int i = 0; i < m; ++i) {
    d = a[i] - x - (i > 0 ? b[i - 1] * b[i - 1] / d : 0.0);
    if (d == 0.0) d = -1e-300;  // an exact zero pivot counts as negative
    c += d < 0.0;
  }
  return c;
}

// One Lanczos step per matrix from the tile pass's partials: w = A_d v -
// beta_prev v_prev, alpha = w . v, w -= alpha v, beta = |w|, next v = w /
// beta; then the witness test above.  mthr: m1 of the fp32 cap.
template <typename T>
__global__ __launch_bounds__(kSvThreads) void lanczos_reduce_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs,
                                                                   RootState* __restrict__ st, int p, double mthr,
                                                                   int kmax) {
  __shared__ double red[kSvThreads / 64];
  __shared__ double sa[kLanczosMax], sb[kLanczosMax];
  const int j = blockIdx.x;
  if (j >= njobs || st[j].status != kActive || st[j].lz_done) return;
  const NewtonJob<T>* J = jobs + j;
  const int n = J->n, TN = J->tiles_n;
  double* v = J->vec;
  double* prow = J->vec + n;
  double* pcol = J->vec + n + (int64_t)TN * n;
  double* vp = J->vec + n + 2 * (int64_t)TN * n;
  double* al = vp + n;
  double* be = al + kLanczosMax;
  const double e = st[j].eps_eff, bprev = st[j].lz_beta;
  const int k = st[j].lz_steps;
  double q = 0.0;
  for (int i = threadIdx.x; i < n; i += kSvThreads) {
    double a = 0.0, b = 0.0;
    for (int c = 0; c < TN; ++c) {
      a += prow[(int64_t)c * n + i];
      b += pcol[(int64_t)c * n + i];
    }
    const double w = 0.5 * (a + b) + e * v[i] - bprev * vp[i];
    prow[i] = w;  // row partials of tile column 0 are consumed: reuse as w
    q += w * v[i];
  }
  const double alpha = sv_block_sum(q, red);
  double s2 = 0.0;
  for (int i = threadIdx.x; i < n; i += kSvThreads) {
    const double w = prow[i] - alpha * v[i];
    prow[i] = w;
    s2 += w * w;
  }
  const double beta = sqrt(sv_block_sum(s2, red));
  for (int i = threadIdx.x; i < n; i += kSvThreads) {
    vp[i] = v[i];
    v[i] = beta > 0.0 ? prow[i] / beta : 0.0;
  }
  for (int i = threadIdx.x; i < k; i += kSvThreads) {
    sa[i] = al[i];
    sb[i] = be[i];
  }
  __shared__ double slo, shi;
  __shared__ int sfirst;
  if (threadIdx.x == 0) {
    sa[k] = alpha;
    al[k] = alpha;
    be[k] = beta;
  }
  __syncthreads();
  const int m = k + 1;
  // smallest Ritz value: the Gershgorin interval, narrowed by three rounds of
  // multisection (every thread counts the eigenvalues below its own point)
  if (threadIdx.x == 0) {
    double lo = INFINITY, hi = -INFINITY;
    for (int i = 0; i < m; ++i) {
      const double r = (i > 0 ? fabs(sb[i - 1]) : 0.0) + (i + 1 < m ? fabs(sb[i]) : 0.0);
      lo = fmin(lo, sa[i] - r);
      hi = fmax(hi, sa[i] + r);
    }
    slo = lo;
    shi = hi;
  }
  for (int round = 0; round < 3; ++round) {
    if (threadIdx.x == 0) sfirst = kSvThreads;
    __syncthreads();
    const double lo = slo, w = (shi - slo) / kSvThreads;
    const double x = lo + w * (threadIdx.x + 1);
    if (sturm_below(sa, sb, m, x) >= 1) atomicMin(&sfirst, (int)threadIdx.x);
    __syncthreads();
    if (threadIdx.x == 0) {
      const int f = sfirst < kSvThreads ? sfirst : kSvThreads - 1;
      slo = lo + w * f;
      shi = lo + w * (f + 1);
    }
    __syncthreads();
  }
  if (threadIdx.x != 0) return;
  const double theta = shi;
  const double top = st[j].lam_max + e;
  const double prev = st[j].lz_theta;
  st[j].lz_steps = m;
  st[j].lz_beta = beta;
  st[j].lz_theta = theta;
  if (theta > 0.0 && top > 0.0 && (p + 1.0) * theta / (2.0 * top) < mthr) {
    st[j].status = kMaxIter;  // certain to end unaccepted in fp32: straight to fp64
    st[j].lz_done = 1;
  } else if (!(theta > 0.0) || beta <= 1e-12 * top || m >= kmax || fabs(prev - theta) <= 1e-2 * theta) {
    st[j].lz_done = 1;
  }
}

// Symmetrised tile pass: thread sees s = (A[r][c] + A[c][r]) / 2 for its
// elements of tile (ti, tj); the transposed block is staged through LDS so
// both reads are coalesced (16-byte loads when the tile is full and aligned).
// Computing a tile and its mirror separately keeps the result exactly
// symmetric because fl(x + y) = fl(y + x).
template <typename F>
__device__ __forceinline__ void sym_tile_pass(const float* __restrict__ A, int n, int ti, int tj,
                                              float* lds /* 128 x 33 */, F&& f) {
  const int r0 = ti * kTile, c0 = tj * kTile;
  const int tid = threadIdx.x;
  const bool vec = (n & 3) == 0 && r0 + kTile <= n && c0 + kTile <= n && (reinterpret_cast<uintptr_t>(A) & 15) == 0;
  for (int q = 0; q < kTile; q += 32) {  // 32-row slab of the tile
    __syncthreads();
    // lds[c][rr] = A[c0 + c][r0 + q + rr]
    if (vec) {
      for (int e = tid; e < kTile * 8; e += kThreads) {
        const int c = e >> 3, rr = (e & 7) * 4;
        const f4v v = gload<f4v>(A + (int64_t)(c0 + c) * n + r0 + q + rr);
#pragma unroll
        for (int k = 0; k < 4; ++k) lds[c * 33 + rr + k] = v[k];
      }
    } else {
      for (int e = tid; e < kTile * 32; e += kThreads) {
        const int c = e >> 5, rr = e & 31;
        const int gr = c0 + c, gc = r0 + q + rr;
        lds[c * 33 + rr] = (gr < n && gc < n) ? A[(int64_t)gr * n + gc] : 0.f;
      }
    }
    __syncthreads();
    if (vec) {
      for (int e = tid; e < 32 * 32; e += kThreads) {
        const int rr = e >> 5, c = (e & 31) * 4;
        const int r = r0 + q + rr;
        const f4v v = gload<f4v>(A + (int64_t)r * n + c0 + c);
#pragma unroll
        for (int k = 0; k < 4; ++k) f(r, c0 + c + k, 0.5 * ((double)v[k] + (double)lds[(c + k) * 33 + rr]));
      }
    } else {
      for (int e = tid; e < 32 * kTile; e += kThreads) {
        const int rr = e >> 7, c = e & 127;
        const int r = r0 + q + rr, cc = c0 + c;
        if (r < n && cc < n) {
          const double s = 0.5 * ((double)A[(int64_t)r * n + cc] + (double)lds[c * 33 + rr]);
          f(r, cc, s);
        }
      }
    }
  }
}

// Per upper tile (ti <= tj): sum of s^2 over the tile, doubled off the
// diagonal (the lower mirror has the same values), trace and minimum of the
// diagonal.  Every element of A is read once from memory.
template <typename T>
__global__ __launch_bounds__(kThreads) void frob_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs,
                                                       const RootState* __restrict__ st, int total_up) {
  __shared__ float lds[kTile * 33];
  __shared__ double red[kThreads / 64];
  const int t = blockIdx.x;
  if (t >= total_up) return;
  const int j = find_job_up(jobs, njobs, t);
  if (st[j].status != kActive) return;
  const NewtonJob<T> J = jobs[j];
  const int lt = t - J.up_begin;
  int ti, tj;
  unrank_upper(lt, J.tiles_n, ti, tj);
  double ss = 0.0, tr = 0.0, dmin = INFINITY;
  sym_tile_pass(J.A, J.n, ti, tj, lds, [&](int r, int c, double s) {
    ss += s * s;
    if (r == c) { tr += s; dmin = dmin < s ? dmin : s; }
  });
  if (ti != tj) ss *= 2.0;
  ss = block_sum(ss, red);
  tr = block_sum(tr, red);
  // min over the block
  double m = dmin;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) { const double w = __shfl_xor(m, o, 64); m = m < w ? m : w; }
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    double mm = red[0];
    for (int w = 1; w < kThreads / 64; ++w) mm = mm < red[w] ? mm : red[w];
    J.part[3 * lt + 0] = ss;
    J.part[3 * lt + 1] = tr;
    J.part[3 * lt + 2] = mm;
  }
}

// One thread per matrix: ||A_d||_F^2 = sum s^2 + 2 eps tr + n eps^2 from the
// tile partials (fixed order), z, NOT_PD check.
template <typename T>
__global__ void root_prep_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs, RootState* __restrict__ st,
                                 int p, int eps_relative, double eps) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= njobs || st[j].status != kActive) return;
  const NewtonJob<T> J = jobs[j];
  const int nt = J.tiles_n * (J.tiles_n + 1) / 2;  // upper-tile partials
  double ss = 0.0, tr = 0.0, dmin = INFINITY;
  for (int q = 0; q < nt; ++q) {
    ss += J.part[3 * q + 0];
    tr += J.part[3 * q + 1];
    const double m = J.part[3 * q + 2];
    dmin = dmin < m ? dmin : m;
  }
  const double e = eps_relative ? st[j].eps_eff : eps;
  if (!eps_relative) st[j].eps_eff = eps;
  const double fro2 = ss + 2.0 * e * tr + (double)J.n * e * e;
  st[j].diag_min = dmin + e;
  if (!(dmin + e > 0.0) || !(fro2 > 0.0) || !isfinite(fro2)) {
    st[j].status = kNotPD;
    st[j].z = 0.0;
    return;
  }
  st[j].z = (1.0 + p) / (2.0 * sqrt(fro2));
  st[j].zc = 1.0;
}

// M0 = z (A_s + eps I), X0 = z^(1/p) I (Algorithm 1 cold start); residual of
// M0 accumulated into resid_bits.  One workgroup per tile of the full grid
// (a version over upper tiles that wrote each tile and its mirror was
// measured slower).
template <typename T>
__global__ __launch_bounds__(kThreads) void root_init_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs,
                                                            RootState* __restrict__ st, int total_full, int p,
                                                            int write_x) {
  __shared__ float lds[kTile * 33];
  const int t = blockIdx.x;
  if (t >= total_full) return;
  const int j = find_job_full(jobs, njobs, t);
  if (st[j].status != kActive) return;
  const NewtonJob<T> J = jobs[j];
  const int lt = t - J.full_begin;
  const int ti = lt / J.tiles_n, tj = lt % J.tiles_n;
  const double z = st[j].z, e = st[j].eps_eff;
  const T x0 = (T)pow(z, 1.0 / p);
  const T a = (T)(p + 1) / (T)p, b = (T)-1 / (T)p;
  const int n = J.n;
  T* M = J.M[0];
  T* X1 = J.X[1];
  float rmax = 0.f;
  // X0 = z^(1/p) I is not stored: the first iterate X1 = X0 M1 =
  // z^(1/p) (a I + b M0) is written here, so the first iteration needs no X
  // product; a matrix that stops before any iteration gets X0 from the
  // output kernel.
  // write_x == 0: only M0 (the power-bound scaling rescales it later)
  sym_tile_pass(J.A, n, ti, tj, lds, [&](int r, int c, double s) {
    const T m = (T)(z * (s + (r == c ? e : 0.0)));
    M[(int64_t)r * n + c] = m;
    if (write_x) {
      X1[(int64_t)r * n + c] = x0 * (b * m + (r == c ? a : (T)0));
      float d = (float)fabs((double)m - (r == c ? 1.0 : 0.0));
      if (!(d <= 3.0e38f)) d = INFINITY;
      rmax = rmax > d ? rmax : d;
    }
  });
  rmax = wave_max(rmax);
  if ((threadIdx.x & 63) == 0 && rmax > 0.f) atomicMax(&st[j].resid_bits, __float_as_uint(rmax));
}

// Power-bound scaling.  ||M0^4||_F^(1/4) = (sum_i mu_i^8)^(1/8) bounds the
// largest eigenvalue mu_max of M0 = z A_d from above, much more tightly than
// ||M0||_F.  With S1 = M0^4 formed by two products, rho = ||S1||_F^(1/4) and
// c = (p + 1) / (2 rho) >= 1, the start M0 <- c M0 keeps the largest
// eigenvalue at or below (p + 1) / 2 (the margin Algorithm 1 keeps with the
// Frobenius bound) while lifting the whole spectrum towards 1.
//
// Per upper tile: sum of squares of S1 (buffer S[1], exactly symmetric),
// doubled off the diagonal, into part[3 t].
template <typename T>
__global__ __launch_bounds__(kThreads) void frob_s1_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs,
                                                          const RootState* __restrict__ st, int total_up) {
  __shared__ double red[kThreads / 64];
  const int t = blockIdx.x;
  if (t >= total_up) return;
  const int j = find_job_up(jobs, njobs, t);
  if (st[j].status != kActive) return;
  const NewtonJob<T>* J = jobs + j;
  const int lt = t - J->up_begin;
  int ti, tj;
  unrank_upper(lt, J->tiles_n, ti, tj);
  const int n = J->n;
  const T* S = J->S[1];
  const int r0 = ti * kTile, c0 = tj * kTile;
  double ss = 0.0;
  if (sizeof(T) == 4 && (n & 3) == 0 && r0 + kTile <= n && c0 + kTile <= n) {
    for (int e = threadIdx.x; e < kTile * kTile / 4; e += kThreads) {
      const f4v x = gload<f4v>(reinterpret_cast<const float*>(S) + (int64_t)(r0 + (e >> 5)) * n + c0 + 4 * (e & 31));
#pragma unroll
      for (int q = 0; q < 4; ++q) ss += (double)x[q] * (double)x[q];
    }
  } else {
    for (int e = threadIdx.x; e < kTile * kTile; e += kThreads) {
      const int r = r0 + (e >> 7), c = c0 + (e & 127);
      if (r < n && c < n) {
        const double x = (double)S[(int64_t)r * n + c];
        ss += x * x;
      }
    }
  }
  if (ti != tj) ss *= 2.0;
  ss = block_sum(ss, red);
  if (threadIdx.x == 0) J->part[3 * lt + 0] = ss;
}

// One thread per matrix: rho from the tile partials (fixed order), c, z *= c.
template <typename T>
__global__ void root_rescale_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs, RootState* __restrict__ st,
                                    int p) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= njobs || st[j].status != kActive) return;
  const NewtonJob<T>* J = jobs + j;
  const int nt = J->tiles_n * (J->tiles_n + 1) / 2;  // upper-tile partials
  double ss = 0.0;
  for (int q = 0; q < nt; ++q) ss += J->part[3 * q + 0];
  const double rho = pow(ss, 0.125);  // ||S1||_F^(1/4)
  double c = (rho > 0.0 && isfinite(rho)) ? (1.0 + p) / (2.0 * rho) : 1.0;
  c = c > 1.0 ? c : 1.0;  // never looser than the Frobenius bound
  st[j].zc = c;
  st[j].z *= c;
}

// M0 <- c M0 in place, X1 = z^(1/p) (a I + b M0), residual of M0.
template <typename T>
__global__ __launch_bounds__(kThreads) void root_scale_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs,
                                                             RootState* __restrict__ st, int total_full, int p) {
  const int t = blockIdx.x;
  if (t >= total_full) return;
  const int j = find_job_full(jobs, njobs, t);
  if (st[j].status != kActive) return;
  const NewtonJob<T>* J = jobs + j;
  const int lt = t - J->full_begin;
  const int ti = lt / J->tiles_n, tj = lt % J->tiles_n;
  const int n = J->n;
  const T c = (T)st[j].zc;
  const T x0 = (T)pow(st[j].z, 1.0 / p);
  const T a = (T)(p + 1) / (T)p, b = (T)-1 / (T)p;
  T* M = J->M[0];
  T* X1 = J->X[1];
  float rmax = 0.f;
  for (int e = threadIdx.x; e < kTile * kTile; e += kThreads) {
    const int r = ti * kTile + (e >> 7), col = tj * kTile + (e & 127);
    if (r < n && col < n) {
      const int64_t i = (int64_t)r * n + col;
      const T m = c * M[i];
      M[i] = m;
      X1[i] = x0 * (b * m + (r == col ? a : (T)0));
      float d = (float)fabs((double)m - (r == col ? 1.0 : 0.0));
      if (!(d <= 3.0e38f)) d = INFINITY;
      rmax = rmax > d ? rmax : d;
    }
  }
  rmax = wave_max(rmax);
  if ((threadIdx.x & 63) == 0 && rmax > 0.f) atomicMax(&st[j].resid_bits, __float_as_uint(rmax));
}

// First stage of iteration 0 under the power-bound scaling.  Its products
// (other than X M1, whose result the init kernel wrote) are all M M with an
// affine epilogue, and M0^2 = c^2 S0 is known from the bound (S0 held the
// square of the unscaled M0), so the stage is elementwise:
//   C_q = ca_q c^2 S0 + cb_q M + cg_q I.
// Each element is read once and every output written after both are formed
// (a product may write S0 itself).
template <typename T>
__global__ __launch_bounds__(kThreads) void newton_poly0_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs,
                                                               RootState* __restrict__ st, int total_full,
                                                               NewtonStage S) {
  const int t = blockIdx.x;
  if (t >= total_full) return;
  const int j = find_job_full(jobs, njobs, t);
  if (st[j].status != kActive) return;
  const NewtonJob<T>* J = jobs + j;
  const int par = st[j].parity;
  const int lt = t - J->full_begin;
  const int ti = lt / J->tiles_n, tj = lt % J->tiles_n;
  const int n = J->n;
  const T c2 = (T)(st[j].zc * st[j].zc);
  const T* S0 = J->S[0];
  const T* M = newton_buf(J, par, kBufMc);
  const int np = S.nprod;
  T* d0 = newton_buf(J, par, S.q[0].dst);
  T* d1 = np > 1 ? newton_buf(J, par, S.q[1].dst) : nullptr;
  const T a0 = (T)S.q[0].ca, b0 = (T)S.q[0].cb, g0 = (T)S.q[0].cg;
  const T a1 = (T)S.q[1].ca, b1 = (T)S.q[1].cb, g1 = (T)S.q[1].cg;
  const bool r0 = S.q[0].resid != 0, r1 = np > 1 && S.q[1].resid != 0;
  float rmax = 0.f;
  for (int e = threadIdx.x; e < kTile * kTile; e += kThreads) {
    const int r = ti * kTile + (e >> 7), col = tj * kTile + (e & 127);
    if (r < n && col < n) {
      const int64_t i = (int64_t)r * n + col;
      const T m2 = c2 * S0[i], m = M[i];
      const bool dg = r == col;
      const T x0 = a0 * m2 + b0 * m + (dg ? g0 : (T)0);
      const T x1 = a1 * m2 + b1 * m + (dg ? g1 : (T)0);
      d0[i] = x0;
      if (d1) d1[i] = x1;
      float d = 0.f;
      if (r0) d = (float)fabs((double)x0 - (dg ? 1.0 : 0.0));
      if (r1) d = (float)fabs((double)x1 - (dg ? 1.0 : 0.0));
      if (!(d <= 3.0e38f)) d = INFINITY;
      rmax = rmax > d ? rmax : d;
    }
  }
  if (r0 || r1) {
    rmax = wave_max(rmax);
    if ((threadIdx.x & 63) == 0 && rmax > 0.f) atomicMax(&st[j].resid_bits, __float_as_uint(rmax));
  }
}

// Start and first iteration at p = 4 under the power-bound scaling, in one
// elementwise pass over the unscaled M0' (as the init kernel wrote it), with
// M0 = c M0'.  M' = M1^4 M0 is a degree-5 polynomial of M0,
// f(M) = sum_i C(4,i) a^(4-i) b^i M^(i+1), and the even powers
// M0^2 = c^2 S0 and M0^4 = c^4 S1 are known from the bound, so
//   M' = M0' (c (k3 M0^2 + k5 M0^4)) + (k1 M0 + k2 M0^2 + k4 M0^4)
// takes one symmetric product.  This pass writes the right operand
// c (k3 M0^2 + k5 M0^4) into S1, the affine term into S0 (in place: every
// element is read, then written, by one thread), the first iterate
// X1 = z^(1/p) (a I + b M0) and the residual max|M0 - I|.  M0 itself is never
// stored.  All outputs stay exactly symmetric.
template <typename T>
__global__ __launch_bounds__(kThreads) void newton_first4_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs,
                                                                RootState* __restrict__ st, int total_flat,
                                                                double k1, double k2, double k3, double k4,
                                                                double k5) {
  const int t = blockIdx.x;
  if (t >= total_flat) return;
  const int j = find_job_flat(jobs, njobs, t);
  if (st[j].status != kActive) return;
  const NewtonJob<T>* J = jobs + j;
  const int n = J->n;
  const int e0 = (t - J->flat_begin) * kFlatChunk, e1 = min(e0 + kFlatChunk, n * n);
  const double cd = st[j].zc;
  const T c = (T)cd, c2 = (T)(cd * cd), c4 = (T)(cd * cd * cd * cd);
  const T K1 = (T)k1, K2 = (T)k2, K3c = (T)(k3 * cd), K4 = (T)k4, K5c = (T)(k5 * cd);
  const T x0 = (T)pow(st[j].z, 0.25);
  const T a = (T)1.25, b = (T)-0.25;
  T* S0 = J->S[0];
  T* S1 = J->S[1];
  T* X1 = J->X[1];
  const T* M = J->M[0];
  float rmax = 0.f;
  auto one = [&](T mu, T s0, T s1, bool dg, T& e, T& r, T& x) {
    const T m = c * mu, m2 = c2 * s0, m4 = c4 * s1;
    r = K3c * m2 + K5c * m4;
    e = K1 * m + K2 * m2 + K4 * m4;
    x = x0 * (b * m + (dg ? a : (T)0));
    float d = (float)fabs((double)m - (dg ? 1.0 : 0.0));
    if (!(d <= 3.0e38f)) d = INFINITY;
    rmax = rmax > d ? rmax : d;
  };
  if (sizeof(T) == 4 && (n & 3) == 0) {
    for (int i = e0 + 4 * (int)threadIdx.x; i < e1; i += 4 * kThreads) {
      const int r = i / n, col = i - r * n;  // the 4 elements share row r
      const f4v m = gload<f4v>(reinterpret_cast<const float*>(M) + i);
      const f4v s0 = gload<f4v>(reinterpret_cast<const float*>(S0) + i);
      const f4v s1 = gload<f4v>(reinterpret_cast<const float*>(S1) + i);
      f4v eo, ro, xo;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        T ee, rr, xx;
        one((T)m[q], (T)s0[q], (T)s1[q], r == col + q, ee, rr, xx);
        eo[q] = (float)ee;
        ro[q] = (float)rr;
        xo[q] = (float)xx;
      }
      gstore<f4v>(reinterpret_cast<float*>(S0) + i, eo);
      gstore<f4v>(reinterpret_cast<float*>(S1) + i, ro);
      gstore<f4v>(reinterpret_cast<float*>(X1) + i, xo);
    }
  } else {
    for (int i = e0 + (int)threadIdx.x; i < e1; i += kThreads) {
      const int r = i / n, col = i - r * n;
      T ee, rr, xx;
      one(M[i], S0[i], S1[i], r == col, ee, rr, xx);
      S0[i] = ee;
      S1[i] = rr;
      X1[i] = xx;
    }
  }
  rmax = wave_max(rmax);
  if ((threadIdx.x & 63) == 0 && rmax > 0.f) atomicMax(&st[j].resid_bits, __float_as_uint(rmax));
}

// Resets the state of the matrices that take part in a phase.
//   phase 0: every matrix (fresh call), phase 1: fp64 tail of AUTO, only
//   matrices flagged `escalate`.
__global__ void root_reset_kernel(RootState* __restrict__ st, int njobs, int phase, int precision) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= njobs) return;
  RootState& s = st[j];
  if (phase == 0) {
    s.status = kActive;
    s.iters = 0;
    s.iters_fp32 = 0;
    s.escalate = 0;
    s.lam_max = 0.0;
    s.eps_eff = 0.0;
    s.diag_min = 0.0;
    s.z = 0.0;
    s.zc = 1.0;
  } else if (!s.escalate) {
    return;
  } else {
    s.status = kActive;
    s.iters = 0;
  }
  s.parity = 0;
  s.resid_bits = 0u;
  s.resid = INFINITY;
  s.precision = precision;
  if (phase == 0) {
    s.warm = 0;
    s.warm_iters = 0;
    s.grew = 0;
    s.xmax_bits = s.mmax_bits = s.comm_bits = 0u;
  }
}

// Per-iteration state machine, one workgroup.  count[0]: matrices still
// active; count[1]: matrices stopped with a result that is not accepted
// (MAXITER or DIVERGED), which the host reads with count[0] to decide on the
// fp64 tail without another synchronisation.
//   init != 0: evaluates the residual of M0 only.
// esc_thr (AUTO fp32 phase, else NULL): esc_thr[k-1] is the largest residual
// after k iterations of a matrix that can still converge within the phase's
// cap; a matrix above it leaves the phase at once (MAXITER, escalated).
// Ends by building the compact tile list of the matrices still active.
__global__ __launch_bounds__(kThreads) void root_update_kernel(RootState* __restrict__ st, int njobs, int init,
                                                              float tol, int max_iters, int* __restrict__ count,
                                                              const float* __restrict__ esc_thr, int esc_n,
                                                              const uint32_t* __restrict__ tmap,
                                                              const int* __restrict__ ubegin, int diag_last,
                                                              uint32_t* __restrict__ tlist, int* __restrict__ tcount) {
  __shared__ int red[2 * (kThreads / 64)];
  int active = 0, fails = 0;
  for (int j = threadIdx.x; j < njobs; j += kThreads) {
    RootState& s = st[j];
    if (s.status != kActive) {
      fails += s.status == kMaxIter || s.status == kDiverged;
      continue;
    }
    const float r = __uint_as_float(s.resid_bits);
    s.resid_bits = 0u;
    if (init) {
      s.resid = r;
      if (!(r <= kDivergeAt)) s.status = kDiverged;
      else if (r <= tol) s.status = kConverged;
    } else {
      s.parity ^= 1;
      s.iters += 1;
      const float prev = s.resid;
      s.resid = r;
      if (!(r <= kDivergeAt)) s.status = kDiverged;
      else if (r <= tol) s.status = kConverged;
      else if (prev < kStagGate && r >= prev) s.status = kStagnated;
      else if (s.iters >= max_iters) s.status = kMaxIter;
      else if (esc_thr && s.iters <= esc_n && r > esc_thr[s.iters - 1]) s.status = kMaxIter;
    }
    if (s.status == kActive) ++active;
    else fails += s.status == kMaxIter || s.status == kDiverged;
  }
  // block reduce
  int a = active, f = fails;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    a += __shfl_xor(a, o, 64);
    f += __shfl_xor(f, o, 64);
  }
  if ((threadIdx.x & 63) == 0) {
    red[threadIdx.x >> 6] = a;
    red[kThreads / 64 + (threadIdx.x >> 6)] = f;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int sa = 0, sf = 0;
    for (int w = 0; w < kThreads / 64; ++w) {
      sa += red[w];
      sf += red[kThreads / 64 + w];
    }
    count[0] = sa;
    count[1] = sf;
  }
  // the next iteration's tiles (every thread's matrices are final here)
  build_tile_list(st, njobs, tmap, ubegin, diag_last, tlist, tcount);
}

// End of the fp32 phase under AUTO: flag matrices whose fp32 result is not
// accepted; counts them.
__global__ __launch_bounds__(kThreads) void root_escalate_kernel(RootState* __restrict__ st, int njobs,
                                                                int* __restrict__ count) {
  __shared__ int red[kThreads / 64];
  int e = 0;
  for (int j = threadIdx.x; j < njobs; j += kThreads) {
    RootState& s = st[j];
    s.iters_fp32 = s.iters;
    const bool ok = s.status == kConverged || s.status == kStagnated || s.status == kNotPD;
    s.escalate = ok ? 0 : 1;
    e += s.escalate;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) e += __shfl_xor(e, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = e;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int w = 0; w < kThreads / 64; ++w) s += red[w];
    *count = s;
  }
}

// Writes the result into the caller's fp32 X: the final iterate when it sits
// in a workspace buffer (fp32 parity 1, or any fp64 result, rounded), or
// X0 = z^(1/p) I for a matrix that stopped before its first iteration.  Only
// matrices whose result came from this phase are touched (`phase_is_tail`
// selects the fp64 tail of AUTO).
template <typename T>
__global__ __launch_bounds__(kThreads) void root_output_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs,
                                                              const RootState* __restrict__ st, int total_flat,
                                                              int phase_is_tail, int p) {
  const int t = blockIdx.x;
  if (t >= total_flat) return;
  const int j = find_job_flat(jobs, njobs, t);
  const RootState& s = st[j];
  if (phase_is_tail && !s.escalate) return;
  if (!phase_is_tail && s.escalate) return;
  if (s.status == kNotPD) return;
  // a warm result at zero iterations is X0 itself, already the caller's X
  // (fp32) or in the current-X buffer (fp64)
  const bool ident = s.iters == 0 && s.warm != 1;
  if (!ident && sizeof(T) == 4 && s.parity == 0) return;  // already in place
  const NewtonJob<T>* J = jobs + j;
  const T* src = J->X[s.parity];
  float* dst = J->Xout;
  const float x0 = (float)pow(s.z, 1.0 / p);
  const int n = J->n;
  const int e0 = (t - J->flat_begin) * kFlatChunk, e1 = min(e0 + kFlatChunk, n * n);
  if (!ident && sizeof(T) == 4 && (n & 3) == 0) {
    for (int i = e0 + 4 * (int)threadIdx.x; i < e1; i += 4 * kThreads)
      gstore<f4v>(dst + i, gload<f4v>(reinterpret_cast<const float*>(src) + i));
    return;
  }
  for (int i = e0 + (int)threadIdx.x; i < e1; i += kThreads) {
    const int r = i / n, c = i - r * n;
    dst[i] = ident ? (r == c ? x0 : 0.f) : (float)src[i];
  }
}

// Largest m0 in (0, 1] the scalar recurrence m <- ((p+1-m)/p)^p m cannot
// bring to |m - 1| <= tol within k iterations; (1 + p) / (2 m*) bounds the
// damped condition number of a matrix that needed k iterations.
__device__ inline int scalar_iters(double m, int p, double tol, int cap) {
  int k = 0;
  while (fabs(m - 1.0) > tol && k < cap) {
    const double f = (p + 1.0 - m) / p;
    double fp = 1.0;
    for (int q = 0; q < p; ++q) fp *= f;
    m = fp * m;
    ++k;
  }
  return k;
}

template <typename T>
__global__ void root_info_kernel(const NewtonJob<T>* __restrict__ jobs, int njobs, const RootState* __restrict__ st,
                                 int p, float tol, void* __restrict__ info_out) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= njobs) return;
  const RootState& s = st[j];
  // condition estimate from the iteration count
  double kappa = 0.0;
  if ((s.status == kConverged || s.status == kStagnated) && s.warm != 1) {
    const double tl = fmax((double)tol, (double)s.resid);
    double lo = 1e-30, hi = 1.0;  // N(lo) > iters >= N(hi) (N decreasing on (0, 1])
    // only N(m) <= iters is asked: counting stops at iters + 1
    const int cap = s.iters + 1;
    if (scalar_iters(lo, p, tl, cap) <= s.iters) {
      kappa = 1.0;
    } else {
      for (int b = 0; b < 40; ++b) {  // hi / lo = 1e30^(2^-40) < 1 + 1e-10
        const double mid = sqrt(lo * hi);
        if (scalar_iters(mid, p, tl, cap) <= s.iters) hi = mid; else lo = mid;
      }
      kappa = (1.0 + p) / (2.0 * hi);
    }
  }
  int32_t* io = reinterpret_cast<int32_t*>(info_out) + 8 * j;
  float* fo = reinterpret_cast<float*>(io);
  io[0] = s.status;
  io[1] = s.iters;
  io[2] = s.precision;
  io[3] = s.precision == 32 ? s.iters : s.iters_fp32;
  fo[4] = s.resid;
  fo[5] = (float)s.lam_max;
  fo[6] = (float)kappa;
  fo[7] = (float)s.eps_eff;
}

// ============================================================================
// Graft: pass 1 (D update, momentum, per-chunk sums of squares) and pass 2
// (per-block step size, parameter update).  Work is split into chunks of
// whole rows of one block.
// ============================================================================
struct GraftBlock {
  const void* G;
  float* W;
  float* D;
  const float* P;
  float* Mg;
  float* Ps;
  int64_t ld;
  int rows, cols;
  int chunk_begin;
  int nchunks;
  int rows_per_chunk;
  int vec4;  // cols, ld, ldw and pointers allow 4-wide vector access
  // W, D, Mg, Ps rows: row r of the block is row wrows[r] (wrows NULL: r)
  // with stride ldw; rows at or past *count are skipped (count NULL: none).
  const int* wrows;
  const int* count;
  int64_t ldw;
  int64_t wlimit;  // rows of the W/D tensor (a wrows entry outside is skipped)
  // pass 2 reduces the block's norm partials partial[2 (part_begin + q)],
  // q < nparts: pass 1's chunks, or the preconditioning GEMM's output tiles
  // when pass 1 is fused into it
  int part_begin;
  int nparts;
};

__device__ __forceinline__ int find_block_graft(const GraftBlock* b, int nb, int t) {
  int lo = 0, hi = nb - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (b[mid].chunk_begin <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Calls f(ig, iw, w) for the elements of a chunk (rows r0..r1 of a block):
// ig is the offset in G and P, iw the offset in W, D, Mg and Ps; 4-wide
// (w = 4) where the block allows vector access, else scalar (w = 1).  Whole
// rows per chunk keep index arithmetic free of divisions.
template <typename F>
__device__ __forceinline__ void for_chunk(const GraftBlock& B, int r0, int r1, F&& f) {
  if (B.count) r1 = min(r1, *B.count);
  for (int r = r0; r < r1; ++r) {
    int64_t wr = r;
    if (B.wrows) {
      wr = B.wrows[r];
      if (wr < 0 || wr >= B.wlimit) continue;
    }
    const int64_t g0 = (int64_t)r * B.ld, w0 = wr * B.ldw;
    if (B.vec4) {
      const int c4 = B.cols >> 2;
      for (int c = threadIdx.x; c < c4; c += kThreads) f(g0 + 4 * c, w0 + 4 * c, 4);
    } else {
      for (int c = threadIdx.x; c < B.cols; c += kThreads) f(g0 + c, w0 + c, 1);
    }
  }
}

// Graft pass 1: per chunk, the squared norms of the magnitude and direction
// terms (partial[2t], partial[2t+1]) and the state updates.
//   AdaGrad (LAMB = false): D += G o G; magnitude Mg = momentum of
//     D^{-1/2} o G; direction Ps = momentum of P.
//   LARS/LAMB (LAMB = true): magnitude ||W||_F (W before the step);
//     direction Ps = momentum of P, or before the roots Mg = momentum of G.
template <typename SG, bool LAMB = false>
__global__ __launch_bounds__(kThreads) void graft_pass1_kernel(const GraftBlock* __restrict__ blocks, int nb,
                                                              int total_chunks, float beta1, int use_shampoo,
                                                              double* __restrict__ partial) {
  __shared__ double red[kThreads / 64];
  const int t = blockIdx.x;
  if (t >= total_chunks) return;
  const GraftBlock B = blocks[find_block_graft(blocks, nb, t)];
  const int ch = t - B.chunk_begin;
  const int r0 = ch * B.rows_per_chunk;
  const int r1 = min(B.rows, r0 + B.rows_per_chunk);
  const bool mom = beta1 > 0.f;
  float smg = 0.f, sps = 0.f;
  if constexpr (LAMB) {
    for_chunk(B, r0, r1, [&](int64_t i, int64_t iw, int w) {
      float g[4], wv[4], pv[4];
      if (w == 4) {
        G4<SG>::load(B.G, i, g);
        const f4v w4 = gload<f4v>(B.W + iw);
        wv[0] = w4[0]; wv[1] = w4[1]; wv[2] = w4[2]; wv[3] = w4[3];
        if (use_shampoo) {
          const f4v p4 = gload<f4v>(B.P + i);
          pv[0] = p4[0]; pv[1] = p4[1]; pv[2] = p4[2]; pv[3] = p4[3];
        }
      } else {
        g[0] = load_g<SG>(B.G, i);
        wv[0] = gload<float>(B.W + iw);
        if (use_shampoo) pv[0] = gload<float>(B.P + i);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (e >= w) break;
        smg += wv[e] * wv[e];
        float mg = g[e];
        if (mom) { mg = beta1 * B.Mg[iw + e] + (1.f - beta1) * g[e]; B.Mg[iw + e] = mg; }
        if (use_shampoo) {
          float ps = pv[e];
          if (mom) { ps = beta1 * B.Ps[iw + e] + (1.f - beta1) * ps; B.Ps[iw + e] = ps; }
          sps += ps * ps;
        } else {
          sps += mg * mg;
        }
      }
    });
  } else
  for_chunk(B, r0, r1, [&](int64_t i, int64_t iw, int w) {
    float g[4], d[4], pv[4];
    if (w == 4) {
      G4<SG>::load(B.G, i, g);
      const f4v dv = gload<f4v>(B.D + iw);
      d[0] = dv[0]; d[1] = dv[1]; d[2] = dv[2]; d[3] = dv[3];
      if (use_shampoo) {
        const f4v p4 = gload<f4v>(B.P + i);
        pv[0] = p4[0]; pv[1] = p4[1]; pv[2] = p4[2]; pv[3] = p4[3];
      }
    } else {
      g[0] = load_g<SG>(B.G, i);
      d[0] = gload<float>(B.D + iw);
      if (use_shampoo) pv[0] = gload<float>(B.P + i);
    }
    f4v dn;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (e >= w) break;
      const float de = d[e] + g[e] * g[e];
      dn[e] = de;
      const float u = ada_dir(g[e], de);
      float mg = u;
      if (mom) { mg = beta1 * B.Mg[iw + e] + (1.f - beta1) * u; B.Mg[iw + e] = mg; }
      smg += mg * mg;
      if (use_shampoo) {
        float ps = pv[e];
        if (mom) { ps = beta1 * B.Ps[iw + e] + (1.f - beta1) * ps; B.Ps[iw + e] = ps; }
        sps += ps * ps;
      }
    }
    if (w == 4) gstore<f4v>(B.D + iw, dn);
    else gstore<float>(B.D + iw, dn[0]);
  });
  const double a = block_sum((double)smg, red);
  const double b = block_sum((double)sps, red);
  if (threadIdx.x == 0) {
    partial[2 * t + 0] = a;
    partial[2 * t + 1] = b;
  }
}

// Graft pass 2: eta from the block's norms, then W -= eta * direction.
template <typename SG, bool LAMB = false>
__global__ __launch_bounds__(kThreads) void graft_pass2_kernel(const GraftBlock* __restrict__ blocks, int nb,
                                                              int total_chunks, float eta0, float beta1,
                                                              int use_shampoo, const double* __restrict__ partial,
                                                              float* __restrict__ norms) {
  __shared__ double red[kThreads / 64];
  // chunk t of the grid-stride walk (a launch of total_chunks workgroups
  // takes one chunk each)
  for (int t = blockIdx.x; t < total_chunks; t += gridDim.x) {
    const int bi = find_block_graft(blocks, nb, t);
    const GraftBlock B = blocks[bi];
    // the block's norms from its chunk partials, reduced cooperatively in a
    // fixed order (every workgroup of the block gets the same bits)
    double smg = 0.0, sps = 0.0;
    for (int q = threadIdx.x; q < B.nparts; q += kThreads) {
      smg += partial[2 * (B.part_begin + q) + 0];
      sps += partial[2 * (B.part_begin + q) + 1];
    }
    smg = block_sum(smg, red);
    sps = block_sum(sps, red);
    const double nm = sqrt(smg), nps = sqrt(sps);
    double eta;
    if (use_shampoo || LAMB) eta = nps > 0.0 ? (double)eta0 * nm / nps : 0.0;
    else eta = eta0;
    const float etaf = (float)eta;
    const int ch = t - B.chunk_begin;
    if (ch == 0 && threadIdx.x == 0 && norms) {
      norms[3 * bi + 0] = (float)nm;
      norms[3 * bi + 1] = (float)nps;
      norms[3 * bi + 2] = etaf;
    }
    if (etaf == 0.f) continue;
    const int r0 = ch * B.rows_per_chunk;
    const int r1 = min(B.rows, r0 + B.rows_per_chunk);
    const bool mom = beta1 > 0.f;
    // direction: Ps (momentum) or P; before the roots Mg or (at beta1 = 0)
    // D^{-1/2} o G, or G itself for LAMB
    const float* dir = use_shampoo ? (mom ? B.Ps : B.P) : (mom ? B.Mg : nullptr);
    // P is laid out like G; momentum buffers like W
    const int64_t dir_w = use_shampoo && !mom ? 0 : 1;
    for_chunk(B, r0, r1, [&](int64_t i, int64_t iw, int w) {
      float step[4];
      const int64_t id = dir_w ? iw : i;
      if (dir) {
        if (w == 4) {
          const f4v v = gload<f4v>(dir + id);
          step[0] = v[0]; step[1] = v[1]; step[2] = v[2]; step[3] = v[3];
        } else {
          step[0] = gload<float>(dir + id);
        }
      } else if (LAMB) {
        if (w == 4) G4<SG>::load(B.G, i, step);
        else step[0] = load_g<SG>(B.G, i);
      } else {
        float g[4];
        if (w == 4) {
          G4<SG>::load(B.G, i, g);
          const f4v dv = gload<f4v>(B.D + iw);
#pragma unroll
          for (int e = 0; e < 4; ++e) step[e] = ada_dir(g[e], dv[e]);
        } else {
          step[0] = ada_dir(load_g<SG>(B.G, i), gload<float>(B.D + iw));
        }
      }
      if (w == 4) {
        f4v wv = gload<f4v>(B.W + iw);
#pragma unroll
        for (int e = 0; e < 4; ++e) wv[e] -= etaf * step[e];
        gstore<f4v>(B.W + iw, wv);
      } else {
        gstore<float>(B.W + iw, gload<float>(B.W + iw) - etaf * step[0]);
      }
    });
  }
}

// P = G (no root on either side), with up-cast.
template <typename SG>
__global__ __launch_bounds__(kThreads) void copy_g_kernel(const GraftBlock* __restrict__ blocks, int nb,
                                                         int total_chunks) {
  const int t = blockIdx.x;
  if (t >= total_chunks) return;
  const GraftBlock B = blocks[find_block_graft(blocks, nb, t)];
  const int ch = t - B.chunk_begin;
  const int r0 = ch * B.rows_per_chunk;
  const int r1 = min(B.rows, r0 + B.rows_per_chunk);
  const int64_t cnt = (int64_t)(r1 - r0) * B.cols;
  float* P = const_cast<float*>(B.P);
  for (int64_t e = threadIdx.x; e < cnt; e += kThreads) {
    const int r = r0 + (int)(e / B.cols), c = (int)(e % B.cols);
    const int64_t i = (int64_t)r * B.ld + c;
    P[i] = load_g<SG>(B.G, i);
  }
}

}  // namespace shp
