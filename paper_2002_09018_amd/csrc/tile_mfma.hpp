// MFMA tile machinery for gfx950 (CDNA4): one workgroup computes a 128 x 128
// output tile C[m0:m0+128, n0:n0+128] = sum_k opA[m, k] * opB[k, n].
//
// Workgroup: 256 threads = 4 wave64s arranged 2 x 2, each owning a 64 x 64
// sub-tile as a grid of MFMA blocks (fp32: 2 x 2 blocks of 32 x 32 with
// v_mfma_f32_32x32x2_f32; fp64: 4 x 4 blocks of 16 x 16 with
// v_mfma_f64_16x16x4_f64).  Wide tiles (WN = 2, plain fp32 products with both
// operands k-major) are 128 x 256: each wave owns 64 x 128 (2 x 4 blocks),
// and B's stage is 256 columns wide.  The k dimension is streamed through LDS in stages
// of kBK = 16, double-buffered: the global loads of stage s+1 are in flight in
// registers while the MFMAs of stage s run (on interior tiles spread over the
// stage's k-steps, see tile_loop).
//
// Each operand stage is copied into LDS in its global orientation, with
// 16-byte loads and 16-byte LDS stores (no transpose):
//   kLayoutK   the stage is read from storage rows k0..k0+kBK, columns
//              i0..i0+128 (the operand's contraction index is its storage row:
//              B of C = A B, or A of C = A^T B, or any symmetric operand);
//              LDS [k][i], unpadded.
//   kLayoutRow the stage is read from storage rows i0..i0+128, columns
//              k0..k0+kBK (contraction index contiguous: A of C = A B,
//              B of C = A B^T); LDS [i][k] with a 16-byte row pad.
// Within a stage, lane group g (lanes with the same lane / kM) takes the
// contraction indices g*KS .. g*KS+KS-1 over the KS MFMA k-steps (a
// permutation of k shared by both operands, so the sum is unchanged).  A
// kLayoutRow fragment of a lane is then KS consecutive elements, read with
// 16-byte LDS loads one chunk of 4 k-steps at a time (holding a whole
// stage's row fragments cost the statistics GEMM an occupancy step); a
// kLayoutK fragment is one element per k-step.
// Source elements may be fp32, fp64 or bf16 (raw uint16 bits, up-cast
// exactly).  Stages go through registers: full, aligned stages with 16-byte
// loads, others with bounds checks (out-of-range elements are loaded as 0).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace shp {

#ifndef SHP_MIN_WAVES
#define SHP_MIN_WAVES 2
#endif
#ifndef SHP_MIN_WAVES_F64
#define SHP_MIN_WAVES_F64 2
#endif
#ifndef SHP_MIN_WAVES_NEWTON_F32
#define SHP_MIN_WAVES_NEWTON_F32 2
#endif
// Minimum waves per SIMD requested from the register allocator
// (__launch_bounds__ second argument).  Measured per kernel: the grouped
// GEMMs run best at 2 (the allocator then reaches 3-4 waves without
// spilling), the fp32 Newton products at 2 as well (138 registers, 3 waves,
// no spills: +1-2% over asking for 4, which spilled in the epilogue once
// every wave of a diagonal tile computes), fp64 at 2.
constexpr int kMinWaves = SHP_MIN_WAVES;
template <typename T>
struct MinWaves {
  static constexpr int value = sizeof(T) == 8 ? SHP_MIN_WAVES_F64 : SHP_MIN_WAVES_NEWTON_F32;
};

constexpr int kTile = 128;
constexpr int kThreads = 256;
constexpr int kWaveTile = 64;

enum { kLayoutK = 0, kLayoutRow = 1 };

template <typename T>
struct Mfma;

#ifndef SHP_BK_F32
#define SHP_BK_F32 16
#endif

template <>
struct Mfma<float> {
  static constexpr int kBK = SHP_BK_F32;  // k-depth of one LDS stage
  static constexpr int kM = 32;   // MFMA block edge
  static constexpr int kK = 2;    // k-depth of one MFMA
  static constexpr int kAcc = 16; // accumulator elements per lane per block
  typedef float acc_t __attribute__((ext_vector_type(16)));
  static __device__ __forceinline__ acc_t mma(float a, float b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  // Position of accumulator element v of `lane` inside a 32 x 32 block.
  static __device__ __forceinline__ int row(int lane, int v) {
    return (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3);
  }
  static __device__ __forceinline__ int col(int lane) { return lane & 31; }
};

template <>
struct Mfma<double> {
  static constexpr int kBK = 16;
  static constexpr int kM = 16;
  static constexpr int kK = 4;
  static constexpr int kAcc = 4;
  typedef double acc_t __attribute__((ext_vector_type(4)));
  static __device__ __forceinline__ acc_t mma(double a, double b, acc_t c) {
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ int row(int lane, int v) { return v * 4 + (lane >> 4); }
  static __device__ __forceinline__ int col(int lane) { return lane & 15; }
};

// Row pitch (elements) of one LDS stage.  kLayoutK: [k][128] rows read as
// contiguous runs (no pad needed: measured conflict-free).  kLayoutRow:
// [128][kBK] rows padded by 16 bytes, so the 16-byte fragment reads of 8
// consecutive rows fall in distinct banks and every row stays 16-byte aligned.
template <typename T, int LAYOUT, int TW = kTile>
struct Pitch {
  static constexpr int value =
      LAYOUT == kLayoutK ? TW : Mfma<T>::kBK + 16 / (int)sizeof(T);
};

// Elements of one operand stage in LDS (TW: the operand's tile width, 128,
// or 256 for B of a wide tile).
template <typename T, int LAYOUT, int TW = kTile>
struct StageElems {
  static constexpr int value = (LAYOUT == kLayoutK ? Mfma<T>::kBK : TW) * Pitch<T, LAYOUT, TW>::value;
  static_assert(value * (int)sizeof(T) % 16 == 0, "stages must stay 16-byte aligned");
};


template <typename S>
struct SrcVec;
template <>
struct SrcVec<float> {
  typedef float type __attribute__((ext_vector_type(4)));
  static constexpr int n = 4;
};
template <>
struct SrcVec<double> {
  typedef double type __attribute__((ext_vector_type(2)));
  static constexpr int n = 2;
};
template <>
struct SrcVec<uint16_t> {
  typedef uint16_t type __attribute__((ext_vector_type(8)));
  static constexpr int n = 8;
};

template <typename T, typename S>
__device__ __forceinline__ T cvt(S x) { return (T)x; }
template <>
__device__ __forceinline__ float cvt<float, uint16_t>(uint16_t x) {
  return __uint_as_float(((uint32_t)x) << 16);
}
template <>
__device__ __forceinline__ double cvt<double, uint16_t>(uint16_t x) {
  return (double)__uint_as_float(((uint32_t)x) << 16);
}

// Global-memory (address space 1) access: keeps operand loads off the flat
// path, whose completion counter is shared with LDS and would make every LDS
// wait also wait for the prefetch of the next stage.
template <typename V>
__device__ __forceinline__ V gload(const void* p) {
  return *(const __attribute__((address_space(1))) V*)(p);
}
template <typename V>
__device__ __forceinline__ void gstore(void* p, V v) {
  *(__attribute__((address_space(1))) V*)(p) = v;
}

// A matrix operand as stored: row-major, `rows` x `cols`, row stride `ld`.
template <typename S>
struct Operand {
  const S* ptr;
  int64_t ld;
  int rows, cols;
  bool aligned;  // ptr and ld allow 16-byte vector loads
};

// Per-thread staging registers for one operand stage (TW: tile width).
template <typename T, typename S, int LAYOUT, int TW = kTile>
struct Loader {
  typedef typename SrcVec<S>::type V;
  static constexpr int VE = SrcVec<S>::n;
  static constexpr int BK = Mfma<T>::kBK;
  static constexpr int NVEC = BK * TW / VE;
  static constexpr int PER = NVEC / kThreads;
  static constexpr int LDP = Pitch<T, LAYOUT, TW>::value;
  static_assert(NVEC % kThreads == 0, "stage must split evenly over the workgroup");
  V buf[PER];

  // Storage coordinates (relative to the stage origin) of vector slot i.
  static __device__ __forceinline__ void slot(int tid, int i, int& sr, int& sc) {
    const int v = tid + i * kThreads;
    if (LAYOUT == kLayoutK) {
      constexpr int VPR = TW / VE;
      sr = v / VPR;
      sc = (v % VPR) * VE;
    } else {
      constexpr int VPR = BK / VE;
      sr = v / VPR;
      sc = (v % VPR) * VE;
    }
  }

  // Whether the stage with storage origin (r0, c0) lies inside the operand
  // and is 16-byte aligned (plain 16-byte loads, no bounds checks).
  static __device__ __forceinline__ bool full(const Operand<S>& op, int r0, int c0) {
    constexpr int SR = LAYOUT == kLayoutK ? BK : TW;
    constexpr int SC = LAYOUT == kLayoutK ? TW : BK;
    return op.aligned && (r0 + SR <= op.rows) && (c0 + SC <= op.cols);
  }

  // Global -> registers, vector slot i of the stage at (r0, c0): a 16-byte
  // load when `fast`, else element loads with bounds checks.
  __device__ __forceinline__ void load_slot(const Operand<S>& op, int r0, int c0, int tid, int i, bool fast) {
    int sr, sc;
    slot(tid, i, sr, sc);
    if (fast) {
      buf[i] = gload<V>(op.ptr + (int64_t)(r0 + sr) * op.ld + (c0 + sc));
    } else {
      const int gr = r0 + sr;
#pragma unroll
      for (int e = 0; e < VE; ++e) {
        const int gc = c0 + sc + e;
        buf[i][e] = (gr < op.rows && gc < op.cols) ? gload<S>(op.ptr + (int64_t)gr * op.ld + gc) : (S)0;
      }
    }
  }

  // Whole stage: one branch for the stage (a branch per slot makes the
  // compiler wait for each 16-byte load before issuing the next).
  __device__ __forceinline__ void load(const Operand<S>& op, int r0, int c0, int tid) {
    if (full(op, r0, c0)) {
#pragma unroll
      for (int i = 0; i < PER; ++i) load_slot(op, r0, c0, tid, i, true);
    } else {
#pragma unroll
      for (int i = 0; i < PER; ++i) load_slot(op, r0, c0, tid, i, false);
    }
  }

  // Registers -> LDS stage, vector slot i (converted to the compute type).
  __device__ __forceinline__ void store_slot(T* lds, int tid, int i) const {
    int sr, sc;
    slot(tid, i, sr, sc);
    T v[VE];
#pragma unroll
    for (int e = 0; e < VE; ++e) v[e] = cvt<T, S>(buf[i][e]);
    T* dst = lds + sr * LDP + sc;
    if (sizeof(T) == 4) {
      typedef float f4 __attribute__((ext_vector_type(4)));
#pragma unroll
      for (int e = 0; e < VE; e += 4) {
        f4 w = {(float)v[e], (float)v[e + 1], (float)v[e + 2], (float)v[e + 3]};
        *reinterpret_cast<f4*>(reinterpret_cast<float*>(dst) + e) = w;
      }
    } else {
      typedef double d2 __attribute__((ext_vector_type(2)));
#pragma unroll
      for (int e = 0; e < VE; e += 2) {
        d2 w = {(double)v[e], (double)v[e + 1]};
        *reinterpret_cast<d2*>(reinterpret_cast<double*>(dst) + e) = w;
      }
    }
  }

  __device__ __forceinline__ void store(T* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) store_slot(lds, tid, i);
  }
};

// Which MFMA blocks of its 64 x 64 square a wave computes.  On a diagonal
// tile of a symmetric output only the upper triangle is stored: the two
// waves on the diagonal skip their blocks below it, and the upper-right
// square is split by block rows between its own wave and the wave of the
// lower-left square (never stored), so no wave idles.
enum : int { kBlocksAll = 0, kBlocksUpper = 1, kBlocksTopHalf = 2, kBlocksBottomHalf = 3 };

template <int MODE, int NB>
__host__ __device__ constexpr bool block_used(int i, int j) {
  return MODE == kBlocksAll ? true
         : MODE == kBlocksUpper ? i <= j
         : MODE == kBlocksTopHalf ? i < NB / 2
                                  : i >= NB / 2;
}

// The wave's square (row and column offsets inside the 128 x 128 tile) and
// block set.
struct WaveRole {
  int wm, wn, mode;
};
__device__ __forceinline__ WaveRole wave_role(int wave, bool diag, int wn = 1) {
  if (!diag) return {(wave >> 1) * kWaveTile, (wave & 1) * kWaveTile * wn, kBlocksAll};
  if (wave == 0) return {0, 0, kBlocksUpper};
  if (wave == 3) return {kWaveTile, kWaveTile, kBlocksUpper};
  return {0, kWaveTile, wave == 1 ? kBlocksTopHalf : kBlocksBottomHalf};
}

// Accumulators of one wave: an NB x NBJ grid of MFMA blocks covering
// 64 x 64 WN.
template <typename T, int WN = 1>
struct WaveAcc {
  static constexpr int NB = kWaveTile / Mfma<T>::kM;
  static constexpr int NBJ = NB * WN;
  typename Mfma<T>::acc_t c[NB][NBJ];

  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < NB; ++i)
#pragma unroll
      for (int j = 0; j < NBJ; ++j)
#pragma unroll
        for (int v = 0; v < Mfma<T>::kAcc; ++v) c[i][j][v] = (T)0;
  }

  // The MFMA k-steps of one LDS stage (kBK / kK steps) over the wave's
  // NB x NBJ blocks.  hook(s) runs at k-step s, after the fragment reads of
  // step s+1 are issued and before the MFMAs of step s.
  // MODE (kBlocks*): the blocks of the wave's square that are computed.
  template <int LA, int LB, int LDPA, int LDPB, int MODE, typename Hook>
  __device__ __forceinline__ void stage(const T* __restrict__ a, const T* __restrict__ b, int wm0,
                                        int wn0, int lane, Hook&& hook) {
    constexpr int KS = Mfma<T>::kBK / Mfma<T>::kK;  // k-steps per stage
    constexpr int VP = 16 / (int)sizeof(T);         // elements per 16-byte LDS read
    constexpr int S0 = 0, S1 = KS;
    static_assert(KS % VP == 0, "row fragments are read 16 bytes at a time");
    typedef T vec_t __attribute__((ext_vector_type(VP)));
    const int g = lane / Mfma<T>::kM;  // this lane's k group: k = g * KS + s at k-step s
    const int ml = lane % Mfma<T>::kM;
    // kLayoutK fragments: one element per k-step, double-buffered in
    // registers so the reads of step s+1 are issued before the MFMAs of s.
    T fa[2][NB], fb[2][NBJ];
    const T* pa = a + g * KS * LDPA + wm0 + ml;
    const T* pb = b + g * KS * LDPB + wn0 + ml;
    if (LA == kLayoutK) {
#pragma unroll
      for (int i = 0; i < NB; ++i) fa[S0 & 1][i] = pa[S0 * LDPA + i * Mfma<T>::kM];
    }
    if (LB == kLayoutK) {
#pragma unroll
      for (int j = 0; j < NBJ; ++j) fb[S0 & 1][j] = pb[S0 * LDPB + j * Mfma<T>::kM];
    }
    // kLayoutRow fragments: VP k-steps per 16-byte read, read per chunk of
    // VP steps (the registers of one chunk only)
#pragma unroll
    for (int cch = S0 / VP; cch < S1 / VP; ++cch) {
      vec_t ra[LA == kLayoutRow ? NB : 1], rb[LB == kLayoutRow ? NBJ : 1];
      if (LA == kLayoutRow) {
#pragma unroll
        for (int i = 0; i < NB; ++i)
          ra[i] = *reinterpret_cast<const vec_t*>(a + (wm0 + i * Mfma<T>::kM + ml) * LDPA + g * KS + cch * VP);
      }
      if (LB == kLayoutRow) {
#pragma unroll
        for (int j = 0; j < NBJ; ++j)
          rb[j] = *reinterpret_cast<const vec_t*>(b + (wn0 + j * Mfma<T>::kM + ml) * LDPB + g * KS + cch * VP);
      }
#pragma unroll
      for (int e = 0; e < VP; ++e) {
        const int s = cch * VP + e;
        const int cur = s & 1;
        if (s + 1 < S1) {
          if (LA == kLayoutK) {
#pragma unroll
            for (int i = 0; i < NB; ++i) fa[cur ^ 1][i] = pa[(s + 1) * LDPA + i * Mfma<T>::kM];
          }
          if (LB == kLayoutK) {
#pragma unroll
            for (int j = 0; j < NBJ; ++j) fb[cur ^ 1][j] = pb[(s + 1) * LDPB + j * Mfma<T>::kM];
          }
        }
        hook(s);
        if (LA == kLayoutK || LB == kLayoutK) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < NB; ++i)
#pragma unroll
          for (int j = 0; j < NBJ; ++j) {
            if (!block_used<MODE, NB>(i, j)) continue;
            c[i][j] = Mfma<T>::mma(LA == kLayoutRow ? ra[i][e] : fa[cur][i], LB == kLayoutRow ? rb[j][e] : fb[cur][j],
                                   c[i][j]);
          }
        if (LA == kLayoutK || LB == kLayoutK) __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
};

// k-loop over LDS stages of one wave with square (wm0, wn0) and block set
// MODE (each block set is a separate loop, so the wave-uniform choice costs
// no registers inside the loop).  Stages alternate between two buffer pairs; the staging of stage st+1 writes the pair that
// stage st-1 read, which every wave left at the barrier ending stage st-1.
//
// Interior tiles (every stage of both operands full and aligned) stage with
// plain 16-byte loads spread over the k-steps: a thread's i-th load of stage
// st+1 is issued at k-step i of stage st and written to LDS at k-step
// KS - PER + i, so the loads have most of a stage to arrive and the MFMA
// stream carries no branches.  The last stage re-loads itself into the idle
// buffer pair instead of testing for the end.  Other tiles (ragged edges, and
// fp64, whose stages are too short to spread) load a whole stage at its start
// and write it to LDS at its end.
template <int MODE, typename T, typename SA, int LA, typename SB, int LB, int WN = 1>
__device__ __forceinline__ void tile_loop(WaveAcc<T, WN>& acc, const Operand<SA>& A, const Operand<SB>& B, int m0,
                                          int n0, int K, T* a0, T* a1, T* b0, T* b1, int wm0, int wn0) {
  constexpr int BK = Mfma<T>::kBK;
  constexpr int KS = BK / Mfma<T>::kK;
  typedef Loader<T, SA, LA> LdA;
  typedef Loader<T, SB, LB, kTile * WN> LdB;
  constexpr bool kSpread = 2 * LdA::PER <= KS && 2 * LdB::PER <= KS;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  LdA la;
  LdB lb;
  const int nst = (K + BK - 1) / BK;
  auto orgA = [&](int k0, int& r, int& c) {
    if (LA == kLayoutK) { r = k0; c = m0; } else { r = m0; c = k0; }
  };
  auto orgB = [&](int k0, int& r, int& c) {
    if (LB == kLayoutK) { r = k0; c = n0; } else { r = n0; c = k0; }
  };
  int ar, ac, br, bc, ar1, ac1, br1, bc1;
  orgA(0, ar, ac);
  orgB(0, br, bc);
  orgA((nst - 1) * BK, ar1, ac1);
  orgB((nst - 1) * BK, br1, bc1);
  // stages are full from the first to the last one when both ends are
  const bool interior = kSpread && nst > 0 && LdA::full(A, ar, ac) && LdA::full(A, ar1, ac1) &&
                        LdB::full(B, br, bc) && LdB::full(B, br1, bc1);
  la.load(A, ar, ac, tid);
  lb.load(B, br, bc, tid);
  la.store(a0, tid);
  lb.store(b0, tid);
  __syncthreads();
  if (interior) {
    for (int st = 0; st < nst; ++st) {
      const bool odd = st & 1;
      const int nx = min(st + 1, nst - 1);
      orgA(nx * BK, ar, ac);
      orgB(nx * BK, br, bc);
      T* na = odd ? a0 : a1;
      T* nb = odd ? b0 : b1;
      acc.template stage<LA, LB, LdA::LDP, LdB::LDP, MODE>(odd ? a1 : a0, odd ? b1 : b0, wm0, wn0, lane, [&](int s) {
        if (s < LdA::PER) la.load_slot(A, ar, ac, tid, s, true);
        if (s < LdB::PER) lb.load_slot(B, br, bc, tid, s, true);
        if (s >= KS - LdA::PER) la.store_slot(na, tid, s - (KS - LdA::PER));
        if (s >= KS - LdB::PER) lb.store_slot(nb, tid, s - (KS - LdB::PER));
      });
      __syncthreads();
    }
    return;
  }
  for (int st = 0; st < nst; ++st) {
    const bool odd = st & 1;
    const bool more = st + 1 < nst;
    if (more) {
      orgA((st + 1) * BK, ar, ac);
      orgB((st + 1) * BK, br, bc);
      la.load(A, ar, ac, tid);
      lb.load(B, br, bc, tid);
    }
    acc.template stage<LA, LB, LdA::LDP, LdB::LDP, MODE>(odd ? a1 : a0, odd ? b1 : b0, wm0, wn0, lane, [](int) {});
    if (more) {
      la.store(odd ? a0 : a1, tid);
      lb.store(odd ? b0 : b1, tid);
    }
    __syncthreads();
  }
}


// Full k-loop of one 128 x (128 WN) output tile.
//   A: layout LA; kLayoutK reads storage rows k (cols m0..), kLayoutRow
//      reads storage rows m0.. (cols k).
//   B: layout LB; kLayoutK reads storage rows k (cols n0..), kLayoutRow
//      reads storage rows n0.. (cols k).
// diag: diagonal tile of a symmetric output (WN = 1 only); the waves take
// the squares and block sets of wave_role (the epilogue must use the same
// roles).
template <typename T, typename SA, int LA, typename SB, int LB, int WN = 1>
__device__ __forceinline__ void tile_mma(WaveAcc<T, WN>& acc, const Operand<SA>& A, const Operand<SB>& B, int m0,
                                         int n0, int K, T* a0, T* a1, T* b0, T* b1, bool diag = false) {
  static_assert(WN == 1 || WN == 2, "tile width 128 or 256");
  const WaveRole ro = wave_role(threadIdx.x >> 6, WN == 1 && diag, WN);
  if (WN > 1 || ro.mode == kBlocksAll)
    tile_loop<kBlocksAll, T, SA, LA, SB, LB, WN>(acc, A, B, m0, n0, K, a0, a1, b0, b1, ro.wm, ro.wn);
  else if constexpr (WN == 1) {
    if (ro.mode == kBlocksUpper)
      tile_loop<kBlocksUpper, T, SA, LA, SB, LB>(acc, A, B, m0, n0, K, a0, a1, b0, b1, ro.wm, ro.wn);
    else if (ro.mode == kBlocksTopHalf)
      tile_loop<kBlocksTopHalf, T, SA, LA, SB, LB>(acc, A, B, m0, n0, K, a0, a1, b0, b1, ro.wm, ro.wn);
    else
      tile_loop<kBlocksBottomHalf, T, SA, LA, SB, LB>(acc, A, B, m0, n0, K, a0, a1, b0, b1, ro.wm, ro.wn);
  }
}

// Workgroup id -> logical tile index so that consecutive logical tiles land
// on the same XCD (workgroups are dealt round-robin over the 8 XCDs, each
// with its own L2): XCD x receives the contiguous logical range
// [x*q + min(x, r), ...) where nwg = 8q + r.
__host__ __device__ __forceinline__ int xcd_remap(int b, int nwg) {
  const int q = nwg >> 3, r = nwg & 7;
  const int x = b & 7, s = b >> 3;
  return x * q + (x < r ? x : r) + s;
}

// Workgroup id -> logical index over two consecutive parts, [0, n1) and
// [n1, n1 + n2): XCD x runs its contiguous share of the first part (as
// xcd_remap), then its contiguous share of the second; -1 past both.  A
// launch needs 8 (ceil((n1 + n2) / 8) + 1) workgroups, since the two
// shares of one XCD round up separately.
__host__ __device__ __forceinline__ int xcd_split_remap(int b, int n1, int n2) {
  const int x = b & 7;
  int s = b >> 3;
  const int q1 = n1 >> 3, r1 = n1 & 7;
  const int c1 = q1 + (x < r1 ? 1 : 0);
  if (s < c1) return x * q1 + (x < r1 ? x : r1) + s;
  s -= c1;
  const int q2 = n2 >> 3, r2 = n2 & 7;
  if (s >= q2 + (x < r2 ? 1 : 0)) return -1;
  return n1 + x * q2 + (x < r2 ? x : r2) + s;
}

// Workgroup id -> logical index for launches whose tiles differ in cost
// (grouped problems of mixed sizes): chunks of kDealChunk consecutive
// indices are dealt round-robin over the 8 XCDs, so every XCD gets an even
// share of the work while its L2 still sees runs of neighbouring tiles.  A
// bijection on [0, 8 kDealChunk m) for every m: such launches pad their grid
// to a multiple of 8 kDealChunk, and ids mapped past the work return.
constexpr int kDealChunk = 8;
// Workgroup -> tile maps of the grouped GEMM: xcd_remap, deal_chunks, or
// (symmetric problems of one size) xcd_split_remap with the diagonal tiles
// last.
enum { kMapXcd = 0, kMapDeal = 1, kMapDiagLast = 2 };
__host__ __device__ __forceinline__ int deal_chunks(int b) {
  const int x = b & 7, s = b >> 3;
  return ((s / kDealChunk) * 8 + x) * kDealChunk + (s % kDealChunk);
}

// Index t of the upper-triangular tile list of a T x T tile grid (row-major
// over ti, tj >= ti) -> (ti, tj).
__host__ __device__ __forceinline__ void unrank_upper(int t, int T, int& ti, int& tj) {
  int i = 0;
  while (t >= T - i) {
    t -= T - i;
    ++i;
  }
  ti = i;
  tj = i + t;
}

// Index t of the strictly upper tile list of a T x T tile grid (row-major
// over ti, tj > ti) -> (ti, tj).
__host__ __device__ __forceinline__ void unrank_strict_upper(int t, int T, int& ti, int& tj) {
  int i = 0;
  while (t >= T - 1 - i) {
    t -= T - 1 - i;
    ++i;
  }
  ti = i;
  tj = i + 1 + t;
}

template <typename T>
__device__ __forceinline__ T wave_max(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    T w = __shfl_xor(v, o, 64);
    v = v > w ? v : w;
  }
  return v;
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace shp
