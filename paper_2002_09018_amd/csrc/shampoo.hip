// Host side of libshampoo: C ABI, argument checking, table upload, launch
// orchestration of the grouped kernels in kernels.hpp.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <string>
#include <vector>

#include <rocprim/device/device_radix_sort.hpp>
#include <rocprim/device/device_run_length_encode.hpp>
#include <rocprim/device/device_scan.hpp>

#include "embedding.hpp"
#include "kernels.hpp"
#include "shampoo.h"

using namespace shp;

// Scratch of shampoo_graft_noalloc: the block table, then the per-chunk norm
// partials.  Every GPU the library runs on holds its own copy for the life
// of the process.  In host code `scratch` names a host-side stand-in, not a
// device address: host code uses the address hipGetSymbolAddress returns for
// the device (Handle::noalloc_dev), resolved once per handle at creation.
static __device__ __align__(256) unsigned char scratch[SHAMPOO_GRAFT_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDim = 4096;
constexpr int kMaxRootJobs = 1 << 22;  // job index field of the packed tile map
constexpr int kMaxRootOrder = 16;  // largest p of X = A^(-1/p)
constexpr int kMaxEmbEntries = 1 << 26;  // lookup entries of one embedding call
constexpr int kCountRing = 64;  // device/pinned slots (pairs) of per-iteration counts
// count pairs: kCountRing per-iteration slots, the initial residual check, the
// AUTO escalation count
constexpr int kCountInts = 2 * (kCountRing + 2);
// allocation-free graft: table region, then fp64 partial pairs
constexpr int kNoallocMaxBlocks = SHAMPOO_GRAFT_NOALLOC_MAX_BLOCKS;
constexpr int kNoallocMaxChunks = SHAMPOO_GRAFT_NOALLOC_MAX_CHUNKS;
constexpr size_t kNoallocTableBytes = (size_t)kNoallocMaxBlocks * sizeof(GraftBlock);
static_assert(kNoallocTableBytes % 256 == 0, "partials must start 256-byte aligned");
static_assert(kNoallocTableBytes + (size_t)kNoallocMaxChunks * 2 * sizeof(double) <= SHAMPOO_GRAFT_NOALLOC_SCRATCH_BYTES,
              "table and partials must fit the scratch array");

inline int cdiv(int a, int b) { return (a + b - 1) / b; }
inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Key of a host table for the upload cache (a hit is confirmed by memcmp,
// so the hash only filters): four independent multiply-xorshift chains over
// 8-byte words (a table of a few tens of KB hashes in microseconds, where a
// byte-serial chain took tens), then the tail bytes.
uint64_t table_hash(const void* p, size_t n) {
  const unsigned char* c = static_cast<const unsigned char*>(p);
  uint64_t h[4] = {0x243F6A8885A308D3ull, 0x13198A2E03707344ull, 0xA4093822299F31D0ull, 0x082EFA98EC4E6C89ull};
  size_t i = 0;
  for (; i + 32 <= n; i += 32)
    for (int l = 0; l < 4; ++l) {
      uint64_t w;
      memcpy(&w, c + i + 8 * l, 8);
      h[l] = (h[l] ^ w) * 0x9E3779B97F4A7C15ull;
      h[l] ^= h[l] >> 29;
    }
  uint64_t r = h[0] ^ (h[1] << 17 | h[1] >> 47) ^ (h[2] << 31 | h[2] >> 33) ^ (h[3] << 47 | h[3] >> 17);
  for (; i < n; ++i) r = (r ^ c[i]) * 1099511628211ull;
  return r ^ (uint64_t)n;
}

struct TableEntry {
  uint64_t key = 0;
  size_t bytes = 0, cap = 0;
  void* dev = nullptr;
  void* host = nullptr;
  hipEvent_t ev = nullptr;
  uint64_t last = 0;
  bool used = false;
};

struct TimedLaunch {
  int cls;
  hipEvent_t a, b;
};

struct Handle {
  int device = 0;
  std::string err;
  std::vector<TableEntry> cache;
  std::vector<int> pending;  // cache entries referenced by the launches being enqueued
  uint64_t clock = 0;
  void* zbuf = nullptr;  // intermediate G Rr of two-sided preconditioning (grown on demand)
  size_t zbuf_cap = 0;
  void* partial = nullptr;
  size_t partial_cap = 0;
  void* sort_tmp = nullptr;  // rocPRIM temporary storage of the embedding row compaction
  size_t sort_tmp_cap = 0;
  int32_t* pinned = nullptr;  // kCountInts ints
  hipEvent_t poll_ev[2] = {nullptr, nullptr};
  bool timing = false;
  std::vector<TimedLaunch> timed;
  std::vector<hipEvent_t> spare_events;
  // shampoo_graft_noalloc: this device's address of `scratch`, the pinned
  // staging of its block table and the event of the last table copy
  void* noalloc_dev = nullptr;
  GraftBlock* noalloc_host = nullptr;
  hipEvent_t noalloc_ev = nullptr;
  // shampoo_precondition_graft: graft pass 2 of a chunk of blocks runs on
  // `side` while the next chunk's GEMMs run on the caller's stream (both at
  // the default priority); `handoff` orders the two
  hipStream_t side = nullptr;
  hipEvent_t handoff = nullptr;
};

struct DeviceGuard {
  int old = -1;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&old) != hipSuccess) old = -1;
    if (old != dev) (void)hipSetDevice(dev);
  }
  ~DeviceGuard() {
    int cur = -1;
    if (old >= 0 && hipGetDevice(&cur) == hipSuccess && cur != old) (void)hipSetDevice(old);
  }
};

shampoo_status fail(Handle* h, shampoo_status code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  if (h) h->err = buf;
  return code;
}

#define HIP_TRY(h, expr)                                                                   \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess) return fail((h), SHAMPOO_EHIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

#define STATUS_TRY(expr)               \
  do {                                 \
    shampoo_status s_ = (expr);        \
    if (s_ != SHAMPOO_OK) return s_;   \
  } while (0)

// Device copy of a host table, cached by content.  An entry is reused only
// after every launch that referenced it has completed (event per entry).
shampoo_status upload_table(Handle* h, const void* data, size_t bytes, hipStream_t s, const void** out) {
  const uint64_t key = table_hash(data, bytes);
  for (size_t i = 0; i < h->cache.size(); ++i) {
    TableEntry& e = h->cache[i];
    if (e.used && e.key == key && e.bytes == bytes && memcmp(e.host, data, bytes) == 0) {
      e.last = ++h->clock;
      h->pending.push_back((int)i);
      *out = e.dev;
      return SHAMPOO_OK;
    }
  }
  int slot = -1;
  if (h->cache.size() < 64) {
    h->cache.emplace_back();
    slot = (int)h->cache.size() - 1;
    HIP_TRY(h, hipEventCreateWithFlags(&h->cache[slot].ev, hipEventDisableTiming));
  } else {
    uint64_t best = UINT64_MAX;
    for (size_t i = 0; i < h->cache.size(); ++i)
      if (h->cache[i].last < best) { best = h->cache[i].last; slot = (int)i; }
    HIP_TRY(h, hipEventSynchronize(h->cache[slot].ev));
  }
  TableEntry& e = h->cache[slot];
  if (e.cap < bytes) {
    if (e.dev) HIP_TRY(h, hipFree(e.dev));
    if (e.host) HIP_TRY(h, hipHostFree(e.host));
    e.dev = e.host = nullptr;
    const size_t cap = std::max<size_t>(align256(bytes), 4096);
    HIP_TRY(h, hipMalloc(&e.dev, cap));
    HIP_TRY(h, hipHostMalloc(&e.host, cap, hipHostMallocDefault));
    e.cap = cap;
  }
  memcpy(e.host, data, bytes);
  HIP_TRY(h, hipMemcpyAsync(e.dev, e.host, bytes, hipMemcpyHostToDevice, s));
  e.key = key;
  e.bytes = bytes;
  e.used = true;
  e.last = ++h->clock;
  h->pending.push_back(slot);
  *out = e.dev;
  return SHAMPOO_OK;
}

// Marks every table referenced since the last call as in use up to here.
shampoo_status tables_done(Handle* h, hipStream_t s) {
  for (int i : h->pending) HIP_TRY(h, hipEventRecord(h->cache[i].ev, s));
  h->pending.clear();
  return SHAMPOO_OK;
}

shampoo_status grow(Handle* h, void** buf, size_t* cap, size_t bytes, hipStream_t s) {
  if (*cap >= bytes) return SHAMPOO_OK;
  // The old buffer may still be read by queued work of this handle, which is
  // ordered on its stream (one handle per stream).
  HIP_TRY(h, hipStreamSynchronize(s));
  if (*buf) HIP_TRY(h, hipFree(*buf));
  *buf = nullptr;
  *cap = 0;
  const size_t c = align256(bytes + bytes / 4);
  HIP_TRY(h, hipMalloc(buf, c));
  *cap = c;
  return SHAMPOO_OK;
}

hipEvent_t take_event(Handle* h) {
  if (!h->spare_events.empty()) {
    hipEvent_t e = h->spare_events.back();
    h->spare_events.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

template <typename F>
shampoo_status launch(Handle* h, int cls, hipStream_t s, F&& f) {
  hipEvent_t a = nullptr, b = nullptr;
  if (h->timing) {
    a = take_event(h);
    b = take_event(h);
    if (!a || !b) return fail(h, SHAMPOO_EHIP, "hipEventCreate failed");
    HIP_TRY(h, hipEventRecord(a, s));
  }
  f();
  HIP_TRY(h, hipGetLastError());
  if (h->timing) {
    HIP_TRY(h, hipEventRecord(b, s));
    h->timed.push_back({cls, a, b});
  }
  return SHAMPOO_OK;
}

template <typename K>
shampoo_status set_lds(Handle* h, K kernel, int bytes) {
  HIP_TRY(h, hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                 hipFuncAttributeMaxDynamicSharedMemorySize, bytes));
  return SHAMPOO_OK;
}

// ---------------------------------------------------------------- GEMM
// Diagonal tiles of a symmetric product launch (the Newton products through
// build_tile_list, the statistics GEMM through kMapDiagLast) run last when
// each XCD has at most this many of them: the cheaper tiles then end
// each XCD's run and even out when its compute units finish, worth a
// fraction of a tile's time per launch.  Measured on uniform launches: with
// up to about 100 per XCD (96 or 62 matrices of 1024 or 512) the launches
// ran 1.8-2.8% faster; from about 150 per XCD on (150 or 576 of 1024, 384
// of 512) they ran up to 2% slower, since each moved tile reads its panels
// again long after the tiles of its row read them, and that cost grows with
// the launch while the gain at its end does not.  Launches of matrices of
// different sizes keep one part.
constexpr int kDiagLastMaxPerXcd = 128;
// The statistics GEMM takes that order at any size once its contraction is
// this deep: measured with G of 2048 or 4096 columns over 192 to 576 blocks,
// 0.8-5% faster, while 1024-deep launches of 144 or 288 blocks ran up to 2%
// slower.  With the cheaper tiles out of the way the early tiles all cost
// the same, so the workgroups of a round start and finish together and
// share the slabs of G they read in L2.
constexpr int kDiagLastMinK = 2048;

template <typename SA, int LA, typename SB, int LB, bool LIM = false, typename SGG = void, int WN = 1>
shampoo_status run_gemm(Handle* h, std::vector<GemmProblem>& probs, hipStream_t s, int cls) {
  if (probs.empty()) return SHAMPOO_OK;
  int total = 0, mixed = 0, sym = 1;
  for (auto& p : probs) {
    p.tiles_n = cdiv(p.N, kTile * WN);  // WN = 2: 256-wide tile columns (plain outputs only)
    p.tile_begin = total;
    total += p.sym ? p.tiles_n * (p.tiles_n + 1) / 2 : cdiv(p.M, kTile) * p.tiles_n;
    mixed |= p.M != probs[0].M || p.N != probs[0].N || p.K != probs[0].K;
    sym &= p.sym;
  }
  // problems of different sizes: tiles dealt in chunks over the XCDs (grid
  // padded to a multiple of 8 chunks); the LIM instantiation keeps dispatch
  // order; symmetric problems of one size, deep or with few diagonal tiles:
  // those last
  const int ndiag = (int)probs.size() * probs[0].tiles_n;
  const bool diag_last = sym && (probs[0].K >= kDiagLastMinK || ndiag <= 8 * kDiagLastMaxPerXcd);
  const int map = LIM ? kMapXcd : mixed ? kMapDeal : diag_last ? kMapDiagLast : kMapXcd;
  const int grid = map == kMapDeal       ? cdiv(total, 8 * kDealChunk) * 8 * kDealChunk
                   : map == kMapDiagLast ? 8 * (cdiv(total, 8) + 1)
                                         : total;
  const void* d = nullptr;
  STATUS_TRY(upload_table(h, probs.data(), probs.size() * sizeof(GemmProblem), s, &d));
  auto k = gemm_grouped_kernel<SA, LA, SB, LB, LIM, SGG, WN>;
  const int lds = 0;  // static LDS
  const int np = (int)probs.size();
  STATUS_TRY(launch(h, cls, s, [&] {
    hipLaunchKernelGGL(k, dim3(grid), dim3(kThreads), lds, s, (const GemmProblem*)d, np, total, map);
  }));
  return SHAMPOO_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

shampoo_status check_blocks(Handle* h, const shampoo_block* blocks, int nblocks, int g_dtype) {
  if (nblocks < 0) return fail(h, SHAMPOO_EINVAL, "nblocks < 0");
  if (nblocks > 0 && !blocks) return fail(h, SHAMPOO_EINVAL, "blocks is NULL");
  if (g_dtype != SHAMPOO_F32 && g_dtype != SHAMPOO_BF16) return fail(h, SHAMPOO_EINVAL, "bad g_dtype %d", g_dtype);
  for (int i = 0; i < nblocks; ++i) {
    const shampoo_block& b = blocks[i];
    if (b.rows < 1 || b.rows > kMaxDim || b.cols < 1 || b.cols > kMaxDim)
      return fail(h, SHAMPOO_EINVAL, "block %d: size %d x %d outside [1, %d]", i, b.rows, b.cols, kMaxDim);
    if (b.ld < b.cols) return fail(h, SHAMPOO_EINVAL, "block %d: ld %lld < cols %d", i, (long long)b.ld, b.cols);
    if (!b.G) return fail(h, SHAMPOO_EINVAL, "block %d: G is NULL", i);
  }
  return SHAMPOO_OK;
}

template <typename SG>
shampoo_status stats_impl(Handle* h, const shampoo_block* blocks, int nb, float beta2, hipStream_t s) {
  const float c = beta2 == 1.0f ? 1.0f : 1.0f - beta2;
  const int ve = 16 / (int)sizeof(SG);
  std::vector<GemmProblem> left, right;
  for (int i = 0; i < nb; ++i) {
    const shampoo_block& b = blocks[i];
    const bool al = aligned16(b.G) && (b.ld % ve) == 0;
    if (b.L) {
      GemmProblem p{};
      p.A = b.G; p.B = b.G; p.C = b.L;
      p.lda = p.ldb = b.ld; p.ldc = b.rows;
      p.a_rows = p.b_rows = b.rows; p.a_cols = p.b_cols = b.cols;
      p.M = p.N = b.rows; p.K = b.cols;
      p.alpha = c; p.beta = beta2; p.sym = 1;
      p.a_aligned = p.b_aligned = al;
      left.push_back(p);
    }
    if (b.R) {
      GemmProblem p{};
      p.A = b.G; p.B = b.G; p.C = b.R;
      p.lda = p.ldb = b.ld; p.ldc = b.cols;
      p.a_rows = p.b_rows = b.rows; p.a_cols = p.b_cols = b.cols;
      p.M = p.N = b.cols; p.K = b.rows;
      p.alpha = c; p.beta = beta2; p.sym = 1;
      p.a_aligned = p.b_aligned = al;
      right.push_back(p);
    }
  }
  // L = G G^T: both operands read with k (= column of G) contiguous.
  STATUS_TRY((run_gemm<SG, kLayoutRow, SG, kLayoutRow>(h, left, s, SHAMPOO_KCLASS_STATS)));
  // R = G^T G: both operands read row by row of G (k = row of G).
  STATUS_TRY((run_gemm<SG, kLayoutK, SG, kLayoutK>(h, right, s, SHAMPOO_KCLASS_STATS)));
  return tables_done(h, s);
}

// ---------------------------------------------------------------- elementwise block tables
// Chunks of one block in the graft kernels: whole rows, at most 16384 elements.
inline int graft_rows_per_chunk(int cols) { return std::max(1, 16384 / cols); }

// Fills out[0..nb) with the graft table of the blocks; returns the chunk count.
int fill_graft_table(const shampoo_block* blocks, int nb, GraftBlock* out) {
  int t = 0;
  for (int i = 0; i < nb; ++i) {
    const shampoo_block& b = blocks[i];
    GraftBlock g{};
    g.G = b.G; g.W = b.W; g.D = b.D; g.P = b.P; g.Mg = b.Mg; g.Ps = b.Ps;
    g.ld = b.ld; g.rows = b.rows; g.cols = b.cols;
    g.ldw = b.ld; g.wrows = nullptr; g.count = nullptr; g.wlimit = b.rows;
    g.rows_per_chunk = graft_rows_per_chunk(b.cols);
    g.nchunks = cdiv(b.rows, g.rows_per_chunk);
    // 4-wide access needs every row start 16-byte aligned in every tensor
    // (G: 8-byte for bf16 is enough since it is read 4 elements at a time)
    const bool al = (b.cols % 4) == 0 && (b.ld % 4) == 0;
    auto a16 = [](const void* p) { return p == nullptr || (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
    g.vec4 = al && a16(b.W) && a16(b.D) && a16(b.P) && a16(b.Mg) && a16(b.Ps) &&
             (reinterpret_cast<uintptr_t>(b.G) & 15) == 0;
    g.chunk_begin = t;
    g.part_begin = t;
    g.nparts = g.nchunks;
    t += g.nchunks;
    out[i] = g;
  }
  return t;
}

std::vector<GraftBlock> graft_table(const shampoo_block* blocks, int nb, int* total) {
  std::vector<GraftBlock> v(nb);
  *total = fill_graft_table(blocks, nb, v.data());
  return v;
}

// Group boundaries of shampoo_precondition_graft: cut[0] = 0 < cut[1] < ...
// < cut[k] = nb, contiguous groups of about equal GEMM flops.  Only calls
// whose blocks all have one shape and one root layout are grouped, with at
// least 8 blocks and 2^24 elements: smaller calls have too short a graft
// pass 2 to pay for the extra launches, and with blocks of mixed sizes every
// group's launches end in a longer tail (measured: C5's step 0.5 ms slower).
// Workgroups of a graft pass 2 that runs on the side stream beside the next
// group's preconditioning GEMMs.  One per row chunk (about 6 000 for a
// quarter of C2's blocks) takes compute units from those GEMMs.  Measured
// on the C2 step (three runs each, same box):
//   64 workgroups: 23.41 ms (the pass no longer finishes under the GEMMs);
//   128: 22.34 ms; 256: 22.32 ms; one per chunk: 22.45 ms.
constexpr int kPass2SideGrid = 256;

std::vector<int> precond_groups(const shampoo_block* blocks, int nb) {
  constexpr int kGroups = 4;
  std::vector<double> w(nb);
  double work = 0.0;
  int64_t elems = 0;
  bool uniform = true;
  for (int i = 0; i < nb; ++i) {
    const shampoo_block& b = blocks[i];
    w[i] = (double)b.rows * b.cols * ((b.Lr ? b.rows : 0) + (b.Rr ? b.cols : 0));
    work += w[i];
    elems += (int64_t)b.rows * b.cols;
    uniform = uniform && b.rows == blocks[0].rows && b.cols == blocks[0].cols &&
              !b.Lr == !blocks[0].Lr && !b.Rr == !blocks[0].Rr;
  }
  std::vector<int> cut{0};
  if (uniform && nb >= 8 && elems >= (int64_t(1) << 24)) {
    double acc = 0.0;
    for (int i = 0; i + 1 < nb && (int)cut.size() < kGroups; ++i) {
      acc += w[i];
      if (acc >= work * (double)cut.size() / kGroups) cut.push_back(i + 1);
    }
  }
  cut.push_back(nb);
  return cut;
}

// fuse_graft: the GEMM that writes a block's P also runs graft pass 1 on it
// (D += G o G and the norm partials of every output tile into h->partial),
// and graft pass 2 follows (AdaGrad graft, beta1 = 0, Shampoo direction);
// every block must have a root.
template <typename SG>
shampoo_status precond_impl(Handle* h, const shampoo_block* blocks, int nb, hipStream_t s, bool fuse_graft = false,
                            float eta0 = 0.f, float* norms = nullptr) {
  const int ve = 16 / (int)sizeof(SG);
  std::vector<GemmProblem> g_rr, lr_z, lr_g;
  std::vector<int> g_rr_b, lr_z_b, lr_g_b;  // block of each problem (ascending)
  // graft: per block, the first and the number of norm partials (the P
  // GEMM's output tiles)
  std::vector<int> pbegin(nb), pcount(nb);
  int ptotal = 0;
  // Without the fused graft, the products by Lr (P = Lr G, or Lr Z) run on
  // 128 x 256 tiles when every block with Lr has a width that is a multiple
  // of 256 (C2: 126 -> 132 TFLOP/s; fewer operand bytes per flop).  G Rr, and
  // every GEMM with the fused graft, keep 128 x 128: the wide kernel runs two
  // workgroups per CU, which hides the graft epilogue less than four
  // (measured: no gain).
  bool wide = !fuse_graft;
  for (int i = 0; i < nb; ++i)
    if (blocks[i].Lr && blocks[i].cols % (2 * kTile) != 0) wide = false;
  if (fuse_graft) {
    for (int i = 0; i < nb; ++i) {
      pbegin[i] = ptotal;
      pcount[i] = cdiv(blocks[i].rows, kTile) * cdiv(blocks[i].cols, kTile);
      ptotal += pcount[i];
    }
    STATUS_TRY(grow(h, &h->partial, &h->partial_cap, (size_t)std::max(ptotal, 1) * 2 * sizeof(double), s));
  }
  double* gpart = static_cast<double*>(h->partial);
  auto with_graft = [&](GemmProblem& q, const shampoo_block& b, int i) {
    if (!fuse_graft) return;
    q.gG = b.G; q.gD = b.D; q.ldg = b.ld; q.gpart = gpart; q.part_base = pbegin[i];
  };
  std::vector<shampoo_block> copy;
  size_t zbytes = 0;
  for (int i = 0; i < nb; ++i) {
    const shampoo_block& b = blocks[i];
    if (b.Lr && b.Rr) zbytes += align256((size_t)b.rows * b.cols * sizeof(float));
  }
  if (zbytes) STATUS_TRY(grow(h, &h->zbuf, &h->zbuf_cap, zbytes, s));
  size_t zoff = 0;
  for (int i = 0; i < nb; ++i) {
    const shampoo_block& b = blocks[i];
    const bool gal = aligned16(b.G) && (b.ld % ve) == 0;
    if (b.Lr && b.Rr) {
      float* Z = reinterpret_cast<float*>(static_cast<char*>(h->zbuf) + zoff);
      zoff += align256((size_t)b.rows * b.cols * sizeof(float));
      GemmProblem p{};  // Z = G Rr
      p.A = b.G; p.lda = b.ld; p.a_rows = b.rows; p.a_cols = b.cols; p.a_aligned = gal;
      p.B = b.Rr; p.ldb = b.cols; p.b_rows = b.cols; p.b_cols = b.cols;
      p.b_aligned = aligned16(b.Rr) && (b.cols % 4) == 0;
      p.C = Z; p.ldc = b.cols; p.M = b.rows; p.N = b.cols; p.K = b.cols;
      p.alpha = 1.f; p.beta = 0.f;
      g_rr.push_back(p);
      g_rr_b.push_back(i);
      GemmProblem q{};  // P = Lr Z, Lr symmetric: read k-major
      q.A = b.Lr; q.lda = b.rows; q.a_rows = b.rows; q.a_cols = b.rows;
      q.a_aligned = aligned16(b.Lr) && (b.rows % 4) == 0;
      q.B = Z; q.ldb = b.cols; q.b_rows = b.rows; q.b_cols = b.cols; q.b_aligned = (b.cols % 4) == 0;
      q.C = b.P; q.ldc = b.ld; q.M = b.rows; q.N = b.cols; q.K = b.rows;
      q.alpha = 1.f; q.beta = 0.f;
      with_graft(q, b, i);
      lr_z.push_back(q);
      lr_z_b.push_back(i);
    } else if (b.Rr) {
      GemmProblem p{};  // P = G Rr
      p.A = b.G; p.lda = b.ld; p.a_rows = b.rows; p.a_cols = b.cols; p.a_aligned = gal;
      p.B = b.Rr; p.ldb = b.cols; p.b_rows = b.cols; p.b_cols = b.cols;
      p.b_aligned = aligned16(b.Rr) && (b.cols % 4) == 0;
      p.C = b.P; p.ldc = b.ld; p.M = b.rows; p.N = b.cols; p.K = b.cols;
      p.alpha = 1.f; p.beta = 0.f;
      with_graft(p, b, i);
      g_rr.push_back(p);
      g_rr_b.push_back(i);
    } else if (b.Lr) {
      GemmProblem q{};  // P = Lr G
      q.A = b.Lr; q.lda = b.rows; q.a_rows = b.rows; q.a_cols = b.rows;
      q.a_aligned = aligned16(b.Lr) && (b.rows % 4) == 0;
      q.B = b.G; q.ldb = b.ld; q.b_rows = b.rows; q.b_cols = b.cols; q.b_aligned = gal;
      q.C = b.P; q.ldc = b.ld; q.M = b.rows; q.N = b.cols; q.K = b.rows;
      q.alpha = 1.f; q.beta = 0.f;
      with_graft(q, b, i);
      lr_g.push_back(q);
      lr_g_b.push_back(i);
    } else {
      copy.push_back(b);
    }
  }
  if (fuse_graft) {
    // The blocks go in contiguous groups of about equal GEMM work: the GEMMs
    // of every group run on the caller's stream, and graft pass 2 of a group
    // (HBM-bound) on the handle's side stream, where it overlaps the GEMMs
    // (MFMA-bound) of the next group.  Each block's result is the same as in
    // one group.
    const std::vector<int> cut = precond_groups(blocks, nb);
    const int ngroups = (int)cut.size() - 1;
    size_t ir = 0, iz = 0, ig = 0;  // next problem of each list
    auto take = [](const std::vector<GemmProblem>& v, const std::vector<int>& vb, size_t& i, int end) {
      std::vector<GemmProblem> out;
      while (i < v.size() && vb[i] < end) out.push_back(v[i++]);
      return out;
    };
    for (int c = 0; c < ngroups; ++c) {
      const int b0 = cut[c], nbc = cut[c + 1] - cut[c];
      std::vector<GemmProblem> c_rr = take(g_rr, g_rr_b, ir, b0 + nbc);
      std::vector<GemmProblem> c_z = take(lr_z, lr_z_b, iz, b0 + nbc);
      std::vector<GemmProblem> c_g = take(lr_g, lr_g_b, ig, b0 + nbc);
      STATUS_TRY((run_gemm<SG, kLayoutRow, float, kLayoutK, false, SG>(h, c_rr, s, SHAMPOO_KCLASS_PRECOND)));
      STATUS_TRY((run_gemm<float, kLayoutK, float, kLayoutK, false, SG>(h, c_z, s, SHAMPOO_KCLASS_PRECOND)));
      STATUS_TRY((run_gemm<float, kLayoutK, SG, kLayoutK, false, SG>(h, c_g, s, SHAMPOO_KCLASS_PRECOND)));
      // graft pass 2 over the row chunks of the group's blocks, with the
      // GEMM's per-tile norm partials
      int total = 0;
      std::vector<GraftBlock> tb = graft_table(blocks + b0, nbc, &total);
      for (int i = 0; i < nbc; ++i) {
        tb[i].part_begin = pbegin[b0 + i];
        tb[i].nparts = pcount[b0 + i];
      }
      const void* d = nullptr;
      STATUS_TRY(upload_table(h, tb.data(), tb.size() * sizeof(GraftBlock), s, &d));
      hipStream_t ps = s;
      if (ngroups > 1) {
        HIP_TRY(h, hipEventRecord(h->handoff, s));
        HIP_TRY(h, hipStreamWaitEvent(h->side, h->handoff, 0));
        ps = h->side;
      }
      float* gn = norms ? norms + 3 * b0 : nullptr;
      // beside the next group's GEMMs, a few workgroups walk the chunks
      // (they leave the GEMMs their compute units); the last group's pass 2
      // runs alone, on the whole GPU
      const int grid = c + 1 < ngroups ? std::min(total, kPass2SideGrid) : total;
      STATUS_TRY(launch(h, SHAMPOO_KCLASS_GRAFT, ps, [&] {
        hipLaunchKernelGGL((graft_pass2_kernel<SG, false>), dim3(grid), dim3(kThreads), 0, ps, (const GraftBlock*)d,
                           nbc, total, eta0, 0.f, 1, (const double*)gpart, gn);
      }));
    }
    if (ngroups > 1) {  // the caller's stream continues after the last pass 2
      HIP_TRY(h, hipEventRecord(h->handoff, h->side));
      HIP_TRY(h, hipStreamWaitEvent(s, h->handoff, 0));
    }
    return tables_done(h, s);
  }
  STATUS_TRY((run_gemm<SG, kLayoutRow, float, kLayoutK>(h, g_rr, s, SHAMPOO_KCLASS_PRECOND)));
  if (wide) {
    STATUS_TRY((run_gemm<float, kLayoutK, float, kLayoutK, false, void, 2>(h, lr_z, s, SHAMPOO_KCLASS_PRECOND)));
    STATUS_TRY((run_gemm<float, kLayoutK, SG, kLayoutK, false, void, 2>(h, lr_g, s, SHAMPOO_KCLASS_PRECOND)));
  } else {
    STATUS_TRY((run_gemm<float, kLayoutK, float, kLayoutK>(h, lr_z, s, SHAMPOO_KCLASS_PRECOND)));
    STATUS_TRY((run_gemm<float, kLayoutK, SG, kLayoutK>(h, lr_g, s, SHAMPOO_KCLASS_PRECOND)));
  }
  if (!copy.empty()) {
    int total = 0;
    std::vector<GraftBlock> tb = graft_table(copy.data(), (int)copy.size(), &total);
    const void* d = nullptr;
    STATUS_TRY(upload_table(h, tb.data(), tb.size() * sizeof(GraftBlock), s, &d));
    const int n = (int)tb.size();
    STATUS_TRY(launch(h, SHAMPOO_KCLASS_PRECOND, s, [&] {
      hipLaunchKernelGGL(copy_g_kernel<SG>, dim3(total), dim3(kThreads), 0, s, (const GraftBlock*)d, n, total);
    }));
  }
  return tables_done(h, s);
}

template <typename SG, bool LAMB>
shampoo_status graft_impl(Handle* h, const shampoo_block* blocks, int nb, float eta0, float beta1, int use_shampoo,
                          float* norms, hipStream_t s) {
  int total = 0;
  std::vector<GraftBlock> tb = graft_table(blocks, nb, &total);
  const void* d = nullptr;
  STATUS_TRY(upload_table(h, tb.data(), tb.size() * sizeof(GraftBlock), s, &d));
  STATUS_TRY(grow(h, &h->partial, &h->partial_cap, (size_t)total * 2 * sizeof(double), s));
  double* part = static_cast<double*>(h->partial);
  const GraftBlock* db = static_cast<const GraftBlock*>(d);
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_GRAFT, s, [&] {
    hipLaunchKernelGGL((graft_pass1_kernel<SG, LAMB>), dim3(total), dim3(kThreads), 0, s, db, nb, total, beta1,
                       use_shampoo, part);
  }));
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_GRAFT, s, [&] {
    hipLaunchKernelGGL((graft_pass2_kernel<SG, LAMB>), dim3(total), dim3(kThreads), 0, s, db, nb, total, eta0, beta1,
                       use_shampoo, (const double*)part, norms);
  }));
  return tables_done(h, s);
}

// ---------------------------------------------------------------- roots
struct RootLayout {
  size_t state = 0, counts = 0, tlist = 0, tcount = 0, tlistf = 0, tcountf = 0, total = 0;
  std::vector<size_t> part, vec, f32, f64;  // per job offsets
};

RootLayout root_layout(const shampoo_root_job* jobs, int njobs, int precision) {
  RootLayout L;
  size_t off = 0;
  L.state = off;
  off += align256((size_t)njobs * sizeof(RootState));
  L.counts = off;
  off += align256(kCountInts * sizeof(int));
  // compact tile list of the product launches (one entry per upper tile)
  size_t up = 0, full = 0;
  for (int j = 0; j < njobs; ++j) {
    const size_t T = (size_t)cdiv(jobs[j].n, kTile);
    up += T * (T + 1) / 2;
    full += T * T;
  }
  L.tlist = off;
  off += align256(up * sizeof(uint32_t));
  L.tcount = off;
  off += 256;
  // and of the warm start's full-grid products
  L.tlistf = off;
  off += align256(full * sizeof(uint32_t));
  L.tcountf = off;
  off += 256;
  for (int j = 0; j < njobs; ++j) {
    const size_t n = (size_t)jobs[j].n;
    const size_t T = (size_t)cdiv(jobs[j].n, kTile);
    L.part.push_back(off);
    off += align256(3 * T * T * sizeof(double));
    L.vec.push_back(off);
    // MaxSV: v and the tile partials; the Lanczos witness: its previous
    // vector and the tridiagonal
    off += align256(((2 * T + 2) * n + 2 * kLanczosMax) * sizeof(double));
    L.f32.push_back(off);
    if (precision != SHAMPOO_PRECISION_FP64) off += 5 * align256(n * n * sizeof(float));
    L.f64.push_back(off);
    if (precision != SHAMPOO_PRECISION_FP32) off += 6 * align256(n * n * sizeof(double));
  }
  L.total = off;
  return L;
}

int host_scalar_iters(double m, int p, double tol, int cap) {
  int k = 0;
  while (fabs(m - 1.0) > tol && k < cap) {
    m = pow((p + 1.0 - m) / p, p) * m;
    ++k;
  }
  return k;
}

// Product program of one coupled Newton iteration for a root order p
// (Algorithm 1): X' = X M1 and M' = M1^p M.  M1^p M is formed right to left
// over the bits of p, with P_s = M1^(2^s) and Y_s = M1^(p mod 2^s) M:
//   stage s: Y <- P_s Y if bit s of p is set;  P_(s+1) = P_s P_s if s < top.
// Both products of a stage read only P_s and Y, so they share one launch (the
// X product joins stage 0).  The last Y product writes M' and carries the
// residual.  Buffers for P and intermediate Y are chosen by a small search so
// that no product writes a buffer that its own launch reads or that holds a
// value still needed; X (current) is free from stage 1 on, since the state
// machine always continues from the new iterate.
struct NewtonProgram {
  std::vector<NewtonStage> stages;  // stage 0 includes the X product (q[0])
};

namespace prog {
struct Pick {
  int y, p;
};

bool search(int p, int s, int top, int pbuf, int ybuf, int rem, std::vector<Pick>& out) {
  if (s > top) return true;
  const bool ybit = (p >> s) & 1;
  std::vector<int> ycand, pcand;
  if (ybit) {
    if (rem == 1) ycand = {kBufMn};
    else ycand = {kBufMn, kBufS1, kBufS0, kBufXc};
  } else {
    ycand = {kBufNone};
  }
  if (s < top) pcand = {kBufS0, kBufS1, kBufXc};
  else pcand = {kBufNone};
  const int pread = pbuf >= 0 ? pbuf : kBufMc;
  for (int yd : ycand)
    for (int pd : pcand) {
      bool ok = true;
      int written[2] = {kBufNone, kBufNone};
      int k = 0;
      for (int d : {yd, pd}) {
        if (d == kBufNone) continue;
        if (d == pread || d == ybuf) ok = false;                   // read in this launch / still live
        if (s == 0 && (d == kBufXc || d == kBufMc || d == kBufXn)) ok = false;  // X product's operands
        if (d == written[0]) ok = false;
        written[k++] = d;
      }
      if (!ok) continue;
      out.push_back({yd, pd});
      if (search(p, s + 1, top, pd != kBufNone ? pd : pbuf, yd != kBufNone ? yd : ybuf, rem - (yd != kBufNone),
                 out))
        return true;
      out.pop_back();
    }
  return false;
}
}  // namespace prog

NewtonProd make_prod(int a, int b, int e, int dst, double ca, double cb, double cg, int resid) {
  NewtonProd q{};
  q.a = a;
  q.b = b;
  q.e = e;
  q.dst = dst;
  q.resid = resid;
  q.ca = ca;
  q.cb = cb;
  q.cg = cg;
  return q;
}

bool build_newton_program(int p, NewtonProgram* out) {
  if (p < 1) return false;
  int top = 0;
  while ((p >> (top + 1)) != 0) ++top;
  const int c = __builtin_popcount((unsigned)p);
  std::vector<prog::Pick> picks;
  if (!prog::search(p, 0, top, kBufNone, kBufMc, c, picks)) return false;
  const double a = (p + 1.0) / p, b = -1.0 / p;
  out->stages.clear();
  int pbuf = kBufNone, ybuf = kBufMc;
  for (int s = 0; s <= top; ++s) {
    NewtonStage st{};
    // X' = X M1 = b (X M) + a X
    if (s == 0) st.q[st.nprod++] = make_prod(kBufXc, kBufMc, kBufXc, kBufXn, b, a, 0.0, 0);
    const prog::Pick k = picks[s];
    if (k.y != kBufNone) {
      const int resid = k.y == kBufMn && s == top;
      if (pbuf == kBufNone)  // M1 Y with Y = M: b (M M) + a M
        st.q[st.nprod++] = make_prod(kBufMc, ybuf, kBufMc, k.y, b, a, 0.0, resid);
      else
        st.q[st.nprod++] = make_prod(pbuf, ybuf, kBufNone, k.y, 1.0, 0.0, 0.0, resid);
    }
    if (k.p != kBufNone) {
      if (pbuf == kBufNone)  // M1 M1 = b^2 (M M) + 2ab M + a^2 I
        st.q[st.nprod++] = make_prod(kBufMc, kBufMc, kBufMc, k.p, b * b, 2.0 * a * b, a * a, 0);
      else
        st.q[st.nprod++] = make_prod(pbuf, pbuf, kBufNone, k.p, 1.0, 0.0, 0.0, 0);
    }
    if (k.y != kBufNone) ybuf = k.y;
    if (k.p != kBufNone) pbuf = k.p;
    out->stages.push_back(st);
  }
  return ybuf == kBufMn;
}

// Stage 0 without its X product (first iteration: X1 is written by the init
// kernel).
NewtonStage drop_x(const NewtonStage& s0) {
  NewtonStage r{};
  for (int i = 1; i < s0.nprod; ++i) r.q[r.nprod++] = s0.q[i];
  return r;
}

// Tiles of the product launches: every upper tile (tmap, job-major, job j's
// from ubegin[j]) and the compact list of the matrices still active (tlist;
// tcount[0] tiles, any late diagonal ones after the first tcount[1]),
// rebuilt at the start of a phase and after every iteration.
struct TileLists {
  const uint32_t* tmap;
  const int* ubegin;
  int diag_last;
  uint32_t* tlist;
  int* tcount;
  int mixed;  // matrices of different sizes (tiles dealt in chunks over the XCDs)
};

// One precision phase of the coupled Newton iteration.
template <typename T>
shampoo_status newton_phase(Handle* h, const NewtonJob<T>* djobs, const TileLists& tl, int njobs, RootState* st, int* dcount,
                            int total_up, int total_full, int total_flat, const NewtonProgram& prog, int p,
                            int scaling, float tol,
                            int cap, int poll, int cls, const float* esc_thr, int esc_n, hipStream_t s,
                            int* fails_out = nullptr) {
  // fails_out: set to the number of matrices stopped unaccepted (MAXITER,
  // DIVERGED) when the polled counts showed that every matrix stopped; left
  // untouched otherwise.
  const int lds = 0;  // static LDS
  auto kstage = newton_stage_kernel<T>;
  const bool power = scaling == SHAMPOO_SCALING_POWER4;
  const int nb1 = cdiv(njobs, 64);
  // grid of a product launch of np products per tile (padded for the
  // chunked deal of matrices of different sizes)
  auto pgrid = [&](int np) {
    return tl.mixed ? cdiv(np * total_up, 8 * kDealChunk) * 8 * kDealChunk : 8 * (cdiv(np * total_up, 8) + 1);
  };
  // M0 (and, with the Frobenius scaling, X1 and the residual of M0); the
  // tiles of the matrices that take part in this phase
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
    hipLaunchKernelGGL(tile_list_kernel, dim3(1), dim3(kThreads), 0, s, st, njobs, tl.tmap, tl.ubegin,
                       tl.diag_last, tl.tlist, tl.tcount);
  }));
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
    hipLaunchKernelGGL(root_init_kernel<T>, dim3(total_full), dim3(kThreads), 0, s, djobs, njobs, st, total_full, p,
                       power ? 0 : 1);
  }));
  // p = 4 under the power-bound scaling: the whole first M update is one
  // product M' = M0' (c (k3 M0^2 + k5 M0^4)) + (k1 M0 + k2 M0^2 + k4 M0^4)
  // with the coefficients of (a + b m)^4 m, a = 5/4, b = -1/4
  const bool first4 = power && p == 4;
  if (power) {
    // S0 = M0^2, S1 = S0^2, rho = ||S1||_F^(1/4), M0 <- c M0 with c = (p+1)/(2 rho)
    NewtonStage sq0{}, sq1{};
    sq0.nprod = sq1.nprod = 1;
    sq0.q[0] = make_prod(kBufMc, kBufMc, kBufNone, kBufS0, 1.0, 0.0, 0.0, 0);
    sq1.q[0] = make_prod(kBufS0, kBufS0, kBufNone, kBufS1, 1.0, 0.0, 0.0, 0);
    for (const NewtonStage* S : {&sq0, &sq1}) {
      STATUS_TRY(launch(h, cls, s, [&] {
        hipLaunchKernelGGL(kstage, dim3(pgrid(1)), dim3(kThreads), lds, s, djobs, tl.tlist, tl.tcount, njobs, st, *S,
                           tl.mixed);
      }));
    }
    const double a = 1.25, b = -0.25;
    STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
      hipLaunchKernelGGL(frob_s1_kernel<T>, dim3(total_up), dim3(kThreads), 0, s, djobs, njobs, st, total_up);
      hipLaunchKernelGGL(root_rescale_kernel<T>, dim3(nb1), dim3(64), 0, s, djobs, njobs, st, p);
      if (first4)
        hipLaunchKernelGGL(newton_first4_kernel<T>, dim3(total_flat), dim3(kThreads), 0, s, djobs, njobs, st,
                           total_flat, a * a * a * a, 4.0 * a * a * a * b, 6.0 * a * a * b * b, 4.0 * a * b * b * b,
                           b * b * b * b);
      else
        hipLaunchKernelGGL(root_scale_kernel<T>, dim3(total_full), dim3(kThreads), 0, s, djobs, njobs, st,
                           total_full, p);
    }));
  }
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
    hipLaunchKernelGGL(root_update_kernel, dim3(1), dim3(kThreads), 0, s, st, njobs, 1, tol, cap,
                       dcount + 2 * kCountRing, (const float*)nullptr, 0, tl.tmap, tl.ubegin, tl.diag_last,
                       tl.tlist, tl.tcount);
  }));
  const NewtonStage first0 = drop_x(prog.stages[0]);
  for (int it = 0; it < cap; ++it) {
    for (size_t q = 0; q < prog.stages.size(); ++q) {
      // iteration 0: X1 = z^(1/p) M1 was written by the init kernel
      const NewtonStage& S = (it == 0 && q == 0) ? first0 : prog.stages[q];
      if (first4 && it == 0) {
        // A = the unscaled M0' (Mc), B = S1, E = S0 as the first4 pass left them
        NewtonStage f{};
        f.nprod = 1;
        f.q[0] = make_prod(kBufMc, kBufS1, kBufS0, kBufMn, 1.0, 1.0, 0.0, 1);
        STATUS_TRY(launch(h, cls, s, [&] {
          hipLaunchKernelGGL(kstage, dim3(pgrid(1)), dim3(kThreads), lds, s, djobs, tl.tlist, tl.tcount, njobs, st, f,
                             tl.mixed);
        }));
        break;  // the iteration's remaining stages are folded into this product
      }
      if (power && it == 0 && q == 0) {
        // M0^2 = c^2 S0 is known: the stage is elementwise
        STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
          hipLaunchKernelGGL(newton_poly0_kernel<T>, dim3(total_full), dim3(kThreads), 0, s, djobs, njobs, st,
                             total_full, S);
        }));
        continue;
      }
      STATUS_TRY(launch(h, cls, s, [&] {
        hipLaunchKernelGGL(kstage, dim3(pgrid(S.nprod)), dim3(kThreads), lds, s, djobs, tl.tlist, tl.tcount, njobs,
                           st, S, tl.mixed);
      }));
    }
    const int ring = 2 * (it % kCountRing);
    int* slot = dcount + ring;
    STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
      hipLaunchKernelGGL(root_update_kernel, dim3(1), dim3(kThreads), 0, s, st, njobs, 0, tol, cap, slot, esc_thr,
                         esc_n, tl.tmap, tl.ubegin, tl.diag_last, tl.tlist, tl.tcount);
    }));
    if (poll) {
      HIP_TRY(h, hipMemcpyAsync(h->pinned + ring, slot, 2 * sizeof(int), hipMemcpyDeviceToHost, s));
      HIP_TRY(h, hipEventRecord(h->poll_ev[it & 1], s));
      if (it >= 1) {
        HIP_TRY(h, hipEventSynchronize(h->poll_ev[(it - 1) & 1]));
        const int32_t* c = h->pinned + 2 * ((it - 1) % kCountRing);
        if (c[0] == 0) {
          // every matrix has stopped: the unaccepted ones are final too
          if (fails_out) *fails_out = c[1];
          break;
        }
      }
    }
  }
  return SHAMPOO_OK;
}

// Warm phase (coupled-Newton appendix, warm start): M0 = X0^p A_d from the
// caller's X0, then Algorithm 1's iteration with full products and, after
// every iteration, the commutator monitor max|XM - MX| <= comm_tol max|X|
// max|M|.  X0^p A_d is formed right to left over the bits of p
// (Y <- P_s Y for a set bit s, P_(s+1) = P_s P_s, P_0 = X0, Y_0 = A_d), so A_d
// stays the rightmost factor; the Y products alternate between two buffers
// so that the last one lands in the current M.  Sets *aborted_out to the
// number of matrices handed to the cold start when the polled counts showed
// the phase finished, else leaves it untouched.
template <typename T>
shampoo_status warm_phase(Handle* h, const NewtonJob<T>* djobs, const TileLists& tf, int njobs, RootState* st,
                          int* dcount, int total_full, const NewtonProgram& prog, int p, float tol, float comm_tol,
                          int cap, int poll, int cls, int32_t* warm_out, hipStream_t s, int* aborted_out) {
  auto kdense = newton_dense_kernel<T>;
  auto run = [&](const NewtonStage& S) {
    const int np = S.nprod;
    const int grid = tf.mixed ? cdiv(np * total_full, 8 * kDealChunk) * 8 * kDealChunk : np * total_full;
    return launch(h, cls, s, [&] {
      hipLaunchKernelGGL(kdense, dim3(grid), dim3(kThreads), 0, s, djobs, tf.tlist, tf.tcount, njobs, st, S, tf.mixed);
    });
  };
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
    hipLaunchKernelGGL(warm_init_kernel<T>, dim3(total_full), dim3(kThreads), 0, s, djobs, njobs, st, total_full);
    hipLaunchKernelGGL(tile_list_kernel, dim3(1), dim3(kThreads), 0, s, st, njobs, tf.tmap, tf.ubegin, 0, tf.tlist,
                       tf.tcount);
  }));
  int top = 0;
  while ((p >> (top + 1)) != 0) ++top;
  const int c = __builtin_popcount((unsigned)p);
  int pb = kBufXc, yb = kBufMn, k = 0;
  for (int b = 0; b <= top; ++b) {
    NewtonStage S{};
    int np = kBufNone, ny = kBufNone;
    if ((p >> b) & 1) {
      ++k;
      ny = (c - k) % 2 == 0 ? kBufMc : kBufXn;
      S.q[S.nprod++] = make_prod(pb, yb, kBufNone, ny, 1.0, 0.0, 0.0, k == c);
    }
    if (b < top) {
      np = pb == kBufS0 ? kBufS1 : kBufS0;
      S.q[S.nprod++] = make_prod(pb, pb, kBufNone, np, 1.0, 0.0, 0.0, 0);
    }
    STATUS_TRY(run(S));
    if (ny != kBufNone) yb = ny;
    if (np != kBufNone) pb = np;
  }
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
    hipLaunchKernelGGL(root_warm_update_kernel, dim3(1), dim3(kThreads), 0, s, st, njobs, 1, tol, comm_tol, cap,
                       dcount + 2 * kCountRing, tf.tmap, tf.ubegin, tf.tlist, tf.tcount);
  }));
  // the iteration's program with the monitor reductions: max|X| on the X
  // product, max|M| on the product that writes the next M
  std::vector<NewtonStage> stages = prog.stages;
  for (NewtonStage& S : stages)
    for (int q = 0; q < S.nprod; ++q) {
      if (S.q[q].dst == kBufXn) S.q[q].amax = kAmaxX;
      if (S.q[q].dst == kBufMn) S.q[q].amax = kAmaxM;
    }
  NewtonStage xm{}, comm{};
  xm.nprod = comm.nprod = 1;
  xm.q[0] = make_prod(kBufXn, kBufMn, kBufNone, kBufS0, 1.0, 0.0, 0.0, 0);       // S0 = X' M'
  comm.q[0] = make_prod(kBufMn, kBufXn, kBufS0, kBufNone, 1.0, -1.0, 0.0, 0);    // M' X' - S0
  comm.q[0].amax = kAmaxComm;
  for (int it = 0; it < cap; ++it) {
    for (const NewtonStage& S : stages) STATUS_TRY(run(S));
    STATUS_TRY(run(xm));
    STATUS_TRY(run(comm));
    const int ring = 2 * (it % kCountRing);
    int* slot = dcount + ring;
    STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
      hipLaunchKernelGGL(root_warm_update_kernel, dim3(1), dim3(kThreads), 0, s, st, njobs, 0, tol, comm_tol, cap,
                         slot, tf.tmap, tf.ubegin, tf.tlist, tf.tcount);
    }));
    if (poll) {
      HIP_TRY(h, hipMemcpyAsync(h->pinned + ring, slot, 2 * sizeof(int), hipMemcpyDeviceToHost, s));
      HIP_TRY(h, hipEventRecord(h->poll_ev[it & 1], s));
      if (it >= 1) {
        HIP_TRY(h, hipEventSynchronize(h->poll_ev[(it - 1) & 1]));
        const int32_t* cnt = h->pinned + 2 * ((it - 1) % kCountRing);
        if (cnt[0] == 0) {
          *aborted_out = cnt[1];
          break;
        }
      }
    }
  }
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
    hipLaunchKernelGGL(root_warm_finish_kernel, dim3(cdiv(njobs, 64)), dim3(64), 0, s, st, njobs, warm_out);
  }));
  return SHAMPOO_OK;
}

template <typename T>
std::vector<NewtonJob<T>> newton_table(const shampoo_root_job* jobs, int njobs, char* ws, const RootLayout& L,
                                       int* total_up, int* total_full, int* total_flat) {
  std::vector<NewtonJob<T>> v(njobs);
  int up = 0, full = 0, flat = 0;
  for (int j = 0; j < njobs; ++j) {
    const int n = jobs[j].n;
    const size_t nn = align256((size_t)n * n * sizeof(T));
    NewtonJob<T>& J = v[j];
    J.A = jobs[j].A;
    J.Xout = jobs[j].X;
    J.part = reinterpret_cast<double*>(ws + L.part[j]);
    J.vec = reinterpret_cast<double*>(ws + L.vec[j]);
    char* base = ws + (sizeof(T) == 4 ? L.f32[j] : L.f64[j]);
    if (sizeof(T) == 4) {
      J.X[0] = reinterpret_cast<T*>(jobs[j].X);
      J.X[1] = reinterpret_cast<T*>(base + 0 * nn);
      J.M[0] = reinterpret_cast<T*>(base + 1 * nn);
      J.M[1] = reinterpret_cast<T*>(base + 2 * nn);
      J.S[0] = reinterpret_cast<T*>(base + 3 * nn);
      J.S[1] = reinterpret_cast<T*>(base + 4 * nn);
    } else {
      J.X[0] = reinterpret_cast<T*>(base + 0 * nn);
      J.X[1] = reinterpret_cast<T*>(base + 1 * nn);
      J.M[0] = reinterpret_cast<T*>(base + 2 * nn);
      J.M[1] = reinterpret_cast<T*>(base + 3 * nn);
      J.S[0] = reinterpret_cast<T*>(base + 4 * nn);
      J.S[1] = reinterpret_cast<T*>(base + 5 * nn);
    }
    J.n = n;
    J.tiles_n = cdiv(n, kTile);
    J.up_begin = up;
    J.full_begin = full;
    J.flat_begin = flat;
    up += J.tiles_n * (J.tiles_n + 1) / 2;
    full += J.tiles_n * J.tiles_n;
    flat += cdiv(n * n, kFlatChunk);
  }
  *total_up = up;
  *total_full = full;
  *total_flat = flat;
  return v;
}

// ---------------------------------------------------------------- embeddings
// Workspace of the embedding calls: seven int32 arrays of nnz (sort keys and
// values in and out, run keys, run lengths, run offsets), the run count, the
// chunk partial sums of the compaction (2 rows of dim per chunk of entries),
// and the split-K partial statistics (splits x dim^2 fp32).
struct EmbLayout {
  size_t keys = 0, vals = 0, keys_s = 0, vals_s = 0, uniq = 0, lens = 0, offs = 0, nruns = 0, cpart = 0, part = 0;
  size_t total = 0;
  int splits = 1;
};

EmbLayout emb_layout(int nnz, int dim) {
  EmbLayout L;
  const size_t a = align256((size_t)nnz * sizeof(int32_t));
  size_t off = 0;
  L.keys = off; off += a;
  L.vals = off; off += a;
  L.keys_s = off; off += a;
  L.vals_s = off; off += a;
  L.uniq = off; off += a;
  L.lens = off; off += a;
  L.offs = off; off += a;
  L.nruns = off; off += 256;
  L.cpart = off; off += align256((size_t)cdiv(nnz, kEmbChunk) * 2 * dim * sizeof(float));
  // Split-K of R += U^T U: about 1024 workgroups over the upper tiles of R.
  // The rows of a split are set on the device from the active-row count u
  // (ceil(u / splits) rounded up to the 16-deep k stage).
  const int t = cdiv(dim, kTile);
  const int tiles = t * (t + 1) / 2;
  const int S = std::max(1, std::min(cdiv(1024, tiles), cdiv(nnz, 256)));
  L.splits = S;
  L.part = off;
  if (S > 1) off += (size_t)S * align256((size_t)dim * dim * sizeof(float));
  L.total = off;
  return L;
}

shampoo_status emb_check(Handle* h, int nnz, int dim) {
  if (nnz < 1 || nnz > kMaxEmbEntries) return fail(h, SHAMPOO_EINVAL, "nnz = %d outside [1, %d]", nnz, kMaxEmbEntries);
  if (dim < 1 || dim > kMaxDim) return fail(h, SHAMPOO_EINVAL, "dim = %d outside [1, %d]", dim, kMaxDim);
  return SHAMPOO_OK;
}

shampoo_status graft_check(Handle* h, const shampoo_block* blocks, int nblocks, int g_dtype, float eta0,
                           float beta1, int use_shampoo, bool lamb) {
  STATUS_TRY(check_blocks(h, blocks, nblocks, g_dtype));
  if (!isfinite(eta0)) return fail(h, SHAMPOO_EINVAL, "eta0 is not finite");
  if (!(beta1 >= 0.f && beta1 < 1.f)) return fail(h, SHAMPOO_EINVAL, "beta1 %g outside [0, 1)", (double)beta1);
  for (int i = 0; i < nblocks; ++i) {
    const shampoo_block& b = blocks[i];
    if (!b.W || (!lamb && !b.D)) return fail(h, SHAMPOO_EINVAL, "block %d: W or D is NULL", i);
    if (use_shampoo && !b.P) return fail(h, SHAMPOO_EINVAL, "block %d: P is NULL", i);
    if (beta1 > 0.f && (!b.Mg || (use_shampoo && !b.Ps)))
      return fail(h, SHAMPOO_EINVAL, "block %d: Mg/Ps needed when beta1 > 0", i);
    // the states written (W, D, and Mg, Ps with momentum) are distinct from
    // each other and from the inputs G and P
    const void* outs[4] = {b.W, lamb ? nullptr : b.D, beta1 > 0.f ? b.Mg : nullptr,
                           beta1 > 0.f && use_shampoo ? b.Ps : nullptr};
    for (int a = 0; a < 4; ++a) {
      if (!outs[a]) continue;
      if (outs[a] == b.G || (use_shampoo && outs[a] == b.P))
        return fail(h, SHAMPOO_EINVAL, "block %d: an updated state aliases G or P", i);
      for (int c = a + 1; c < 4; ++c)
        if (outs[a] == outs[c]) return fail(h, SHAMPOO_EINVAL, "block %d: updated states alias", i);
    }
  }
  return SHAMPOO_OK;
}

shampoo_status graft_entry(void* handle, const shampoo_block* blocks, int nblocks, int g_dtype, float eta0,
                           float beta1, int use_shampoo, float* norms, void* stream, bool lamb) {
  Handle* h = static_cast<Handle*>(handle);
  if (!h) return SHAMPOO_EINVAL;
  h->err.clear();
  STATUS_TRY(graft_check(h, blocks, nblocks, g_dtype, eta0, beta1, use_shampoo, lamb));
  if (nblocks == 0) return SHAMPOO_OK;
  DeviceGuard g(h->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (lamb) {
    if (g_dtype == SHAMPOO_F32) return graft_impl<float, true>(h, blocks, nblocks, eta0, beta1, use_shampoo, norms, s);
    return graft_impl<uint16_t, true>(h, blocks, nblocks, eta0, beta1, use_shampoo, norms, s);
  }
  if (g_dtype == SHAMPOO_F32) return graft_impl<float, false>(h, blocks, nblocks, eta0, beta1, use_shampoo, norms, s);
  return graft_impl<uint16_t, false>(h, blocks, nblocks, eta0, beta1, use_shampoo, norms, s);
}

}  // namespace

// ============================================================================
// C ABI
// ============================================================================
extern "C" {

const char* shampoo_version(void) { return "shampoo-mi355x 0.1 (gfx950)"; }

void shampoo_root_params_default(shampoo_root_params* q) {
  if (!q) return;
  q->p = 4;
  q->eps = 1e-6f;
  q->eps_relative = 0;
  q->tol = 1e-6f;
  q->max_iters = 100;
  q->precision = SHAMPOO_PRECISION_AUTO;
  q->kappa32 = 1e4f;
  q->maxsv_steps = 100;
  q->maxsv_tol = 1e-6f;
  q->poll = 1;
  q->scaling = SHAMPOO_SCALING_POWER4;
}

shampoo_status shampoo_create(void** handle, int device) {
  if (!handle) return SHAMPOO_EINVAL;
  *handle = nullptr;
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || device < 0 || device >= ndev) return SHAMPOO_EINVAL;
  Handle* h = new Handle();
  h->device = device;
  DeviceGuard g(device);
  h->err.reserve(512);  // fail() then never reallocates (messages are at most 511 characters)
  if (hipHostMalloc(reinterpret_cast<void**>(&h->pinned), kCountInts * sizeof(int32_t),
                    hipHostMallocDefault) != hipSuccess ||
      hipEventCreateWithFlags(&h->poll_ev[0], hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&h->poll_ev[1], hipEventDisableTiming) != hipSuccess ||
      // set-up of the allocation-free graft, with this device current
      hipGetSymbolAddress(&h->noalloc_dev, HIP_SYMBOL(scratch)) != hipSuccess || !h->noalloc_dev ||
      hipHostMalloc(reinterpret_cast<void**>(&h->noalloc_host), kNoallocTableBytes, hipHostMallocDefault) !=
          hipSuccess ||
      hipEventCreateWithFlags(&h->noalloc_ev, hipEventDisableTiming) != hipSuccess ||
      hipStreamCreateWithFlags(&h->side, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&h->handoff, hipEventDisableTiming) != hipSuccess) {
    if (h->pinned) (void)hipHostFree(h->pinned);
    if (h->noalloc_host) (void)hipHostFree(h->noalloc_host);
    for (auto e : h->poll_ev)
      if (e) (void)hipEventDestroy(e);
    if (h->noalloc_ev) (void)hipEventDestroy(h->noalloc_ev);
    if (h->side) (void)hipStreamDestroy(h->side);
    delete h;
    return SHAMPOO_EHIP;
  }
  *handle = h;
  return SHAMPOO_OK;
}

shampoo_status shampoo_destroy(void* handle) {
  Handle* h = static_cast<Handle*>(handle);
  if (!h) return SHAMPOO_EINVAL;
  DeviceGuard g(h->device);
  (void)hipDeviceSynchronize();
  for (auto& e : h->cache) {
    if (e.dev) (void)hipFree(e.dev);
    if (e.host) (void)hipHostFree(e.host);
    if (e.ev) (void)hipEventDestroy(e.ev);
  }
  for (auto& t : h->timed) {
    (void)hipEventDestroy(t.a);
    (void)hipEventDestroy(t.b);
  }
  for (auto e : h->spare_events) (void)hipEventDestroy(e);
  if (h->zbuf) (void)hipFree(h->zbuf);
  if (h->partial) (void)hipFree(h->partial);
  if (h->sort_tmp) (void)hipFree(h->sort_tmp);
  if (h->pinned) (void)hipHostFree(h->pinned);
  for (auto e : h->poll_ev)
    if (e) (void)hipEventDestroy(e);
  if (h->noalloc_host) (void)hipHostFree(h->noalloc_host);
  if (h->noalloc_ev) (void)hipEventDestroy(h->noalloc_ev);
  if (h->handoff) (void)hipEventDestroy(h->handoff);
  if (h->side) (void)hipStreamDestroy(h->side);
  delete h;
  return SHAMPOO_OK;
}

const char* shampoo_last_error(const void* handle) {
  const Handle* h = static_cast<const Handle*>(handle);
  return h ? h->err.c_str() : "invalid handle";
}

shampoo_status shampoo_update_stats(void* handle, const shampoo_block* blocks, int nblocks, int g_dtype,
                                    float beta2, void* stream) {
  Handle* h = static_cast<Handle*>(handle);
  if (!h) return SHAMPOO_EINVAL;
  h->err.clear();
  STATUS_TRY(check_blocks(h, blocks, nblocks, g_dtype));
  if (!(beta2 > 0.f && beta2 <= 1.f)) return fail(h, SHAMPOO_EINVAL, "beta2 %g outside (0, 1]", (double)beta2);
  for (int i = 0; i < nblocks; ++i) {
    const shampoo_block& b = blocks[i];
    if ((b.L && (b.L == b.G || b.L == b.R)) || (b.R && b.R == b.G))
      return fail(h, SHAMPOO_EINVAL, "block %d: L, R and G must be distinct", i);
  }
  if (nblocks == 0) return SHAMPOO_OK;
  DeviceGuard g(h->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (g_dtype == SHAMPOO_F32) return stats_impl<float>(h, blocks, nblocks, beta2, s);
  return stats_impl<uint16_t>(h, blocks, nblocks, beta2, s);
}

shampoo_status shampoo_precondition(void* handle, const shampoo_block* blocks, int nblocks, int g_dtype,
                                    void* stream) {
  Handle* h = static_cast<Handle*>(handle);
  if (!h) return SHAMPOO_EINVAL;
  h->err.clear();
  STATUS_TRY(check_blocks(h, blocks, nblocks, g_dtype));
  for (int i = 0; i < nblocks; ++i) {
    const shampoo_block& b = blocks[i];
    if (!b.P) return fail(h, SHAMPOO_EINVAL, "block %d: P is NULL", i);
    // the GEMMs read G and the roots while other workgroups write P
    if (b.P == b.G || (const float*)b.P == b.Lr || (const float*)b.P == b.Rr)
      return fail(h, SHAMPOO_EINVAL, "block %d: P aliases G or a root", i);
  }
  if (nblocks == 0) return SHAMPOO_OK;
  DeviceGuard g(h->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (g_dtype == SHAMPOO_F32) return precond_impl<float>(h, blocks, nblocks, s);
  return precond_impl<uint16_t>(h, blocks, nblocks, s);
}

shampoo_status shampoo_graft(void* handle, const shampoo_block* blocks, int nblocks, int g_dtype, float eta0,
                             float beta1, int use_shampoo, float* norms, void* stream) {
  return graft_entry(handle, blocks, nblocks, g_dtype, eta0, beta1, use_shampoo, norms, stream, false);
}

shampoo_status shampoo_graft_noalloc(void* handle, const shampoo_block* blocks, int nblocks, int g_dtype,
                                     float eta0, float beta1, int use_shampoo, float* norms, void* stream) {
  Handle* h = static_cast<Handle*>(handle);
  if (!h) return SHAMPOO_EINVAL;
  h->err.clear();
  STATUS_TRY(graft_check(h, blocks, nblocks, g_dtype, eta0, beta1, use_shampoo, false));
  if (nblocks == 0) return SHAMPOO_OK;
  if (nblocks > kNoallocMaxBlocks)
    return fail(h, SHAMPOO_ENOMEM, "%d blocks exceed the allocation-free graft's limit of %d", nblocks,
                kNoallocMaxBlocks);
  int64_t chunks = 0;
  for (int i = 0; i < nblocks; ++i) chunks += cdiv(blocks[i].rows, graft_rows_per_chunk(blocks[i].cols));
  if (chunks > kNoallocMaxChunks)
    return fail(h, SHAMPOO_ENOMEM, "%lld chunks exceed the allocation-free graft's limit of %d", (long long)chunks,
                kNoallocMaxChunks);
  DeviceGuard g(h->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // the previous call's table copy must have left the staging memory
  HIP_TRY(h, hipEventSynchronize(h->noalloc_ev));
  const int total = fill_graft_table(blocks, nblocks, h->noalloc_host);
  GraftBlock* dtab = static_cast<GraftBlock*>(h->noalloc_dev);
  double* part = reinterpret_cast<double*>(static_cast<char*>(h->noalloc_dev) + kNoallocTableBytes);
  HIP_TRY(h, hipMemcpyAsync(dtab, h->noalloc_host, (size_t)nblocks * sizeof(GraftBlock), hipMemcpyHostToDevice, s));
  HIP_TRY(h, hipEventRecord(h->noalloc_ev, s));
  if (g_dtype == SHAMPOO_F32) {
    hipLaunchKernelGGL((graft_pass1_kernel<float, false>), dim3(total), dim3(kThreads), 0, s, dtab, nblocks, total,
                       beta1, use_shampoo, part);
    hipLaunchKernelGGL((graft_pass2_kernel<float, false>), dim3(total), dim3(kThreads), 0, s, dtab, nblocks, total,
                       eta0, beta1, use_shampoo, (const double*)part, norms);
  } else {
    hipLaunchKernelGGL((graft_pass1_kernel<uint16_t, false>), dim3(total), dim3(kThreads), 0, s, dtab, nblocks,
                       total, beta1, use_shampoo, part);
    hipLaunchKernelGGL((graft_pass2_kernel<uint16_t, false>), dim3(total), dim3(kThreads), 0, s, dtab, nblocks,
                       total, eta0, beta1, use_shampoo, (const double*)part, norms);
  }
  HIP_TRY(h, hipGetLastError());
  return SHAMPOO_OK;
}

shampoo_status shampoo_precondition_graft(void* handle, const shampoo_block* blocks, int nblocks, int g_dtype,
                                         float eta0, float* norms, void* stream) {
  Handle* h = static_cast<Handle*>(handle);
  if (!h) return SHAMPOO_EINVAL;
  h->err.clear();
  STATUS_TRY(check_blocks(h, blocks, nblocks, g_dtype));
  if (!isfinite(eta0)) return fail(h, SHAMPOO_EINVAL, "eta0 is not finite");
  for (int i = 0; i < nblocks; ++i) {
    const shampoo_block& b = blocks[i];
    if (!b.P || !b.W || !b.D) return fail(h, SHAMPOO_EINVAL, "block %d: P, W or D is NULL", i);
    if (!b.Lr && !b.Rr) return fail(h, SHAMPOO_EINVAL, "block %d: no root (use shampoo_graft)", i);
    const void* outs[3] = {b.P, b.W, b.D};
    for (const void* o : outs)
      if (o == b.G || o == (const void*)b.Lr || o == (const void*)b.Rr)
        return fail(h, SHAMPOO_EINVAL, "block %d: P, W or D aliases G or a root", i);
    if (b.P == b.W || b.P == b.D || b.W == b.D)
      return fail(h, SHAMPOO_EINVAL, "block %d: P, W and D must be distinct", i);
  }
  if (nblocks == 0) return SHAMPOO_OK;
  DeviceGuard g(h->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (g_dtype == SHAMPOO_BF16) return precond_impl<uint16_t>(h, blocks, nblocks, s, true, eta0, norms);
  return precond_impl<float>(h, blocks, nblocks, s, true, eta0, norms);
}

shampoo_status shampoo_graft_lamb(void* handle, const shampoo_block* blocks, int nblocks, int g_dtype, float eta0,
                                  float beta1, int use_shampoo, float* norms, void* stream) {
  return graft_entry(handle, blocks, nblocks, g_dtype, eta0, beta1, use_shampoo, norms, stream, true);
}

size_t shampoo_inv_root_workspace_bytes(const shampoo_root_job* jobs, int njobs, int precision) {
  if (njobs < 0 || (njobs > 0 && !jobs)) return 0;
  if (precision < SHAMPOO_PRECISION_FP32 || precision > SHAMPOO_PRECISION_FP64) return 0;
  for (int j = 0; j < njobs; ++j)
    if (jobs[j].n < 1 || jobs[j].n > kMaxDim) return 0;
  return root_layout(jobs, njobs, precision).total;
}

}  // extern "C"

namespace {
// Both root entry points.  warm: the warm start of the coupled-Newton
// appendix from the caller's X, in the precision the policy starts in (fp64
// under FP64, else fp32), with the cold start for the matrices whose warm
// start is given up.
shampoo_status inv_root_impl(Handle* h, const shampoo_root_job* jobs, int njobs, const shampoo_root_params* prm,
                             int warm, float comm_tol, void* workspace, size_t ws_bytes, shampoo_root_info* info,
                             int32_t* warm_out, void* stream) {
  if (!h) return SHAMPOO_EINVAL;
  h->err.clear();
  if (!prm) return fail(h, SHAMPOO_EINVAL, "params is NULL");
  if (warm && !(comm_tol > 0.f)) return fail(h, SHAMPOO_EINVAL, "comm_tol must be > 0");
  if (njobs < 0) return fail(h, SHAMPOO_EINVAL, "njobs < 0");
  if (njobs == 0) return SHAMPOO_OK;
  if (njobs > kMaxRootJobs) return fail(h, SHAMPOO_EINVAL, "njobs = %d above %d", njobs, kMaxRootJobs);
  if (!jobs || !info || !workspace) return fail(h, SHAMPOO_EINVAL, "jobs, info or workspace is NULL");
  const int p = prm->p;
  if (p < 1 || p > kMaxRootOrder) return fail(h, SHAMPOO_EUNSUPPORTED, "p = %d outside [1, %d]", p, kMaxRootOrder);
  NewtonProgram prog;
  if (!build_newton_program(p, &prog)) return fail(h, SHAMPOO_EUNSUPPORTED, "no product program for p = %d", p);
  if (!(prm->eps >= 0.f) || !isfinite(prm->eps)) return fail(h, SHAMPOO_EINVAL, "eps must be finite and >= 0");
  if (!(prm->tol >= 0.f)) return fail(h, SHAMPOO_EINVAL, "tol must be >= 0");
  if (prm->max_iters < 1) return fail(h, SHAMPOO_EINVAL, "max_iters must be >= 1");
  if (prm->precision < 0 || prm->precision > 2) return fail(h, SHAMPOO_EINVAL, "bad precision %d", prm->precision);
  if (prm->eps_relative && prm->maxsv_steps < 1) return fail(h, SHAMPOO_EINVAL, "maxsv_steps must be >= 1");
  if (prm->scaling != SHAMPOO_SCALING_FROBENIUS && prm->scaling != SHAMPOO_SCALING_POWER4)
    return fail(h, SHAMPOO_EINVAL, "bad scaling %d", prm->scaling);
  if (prm->precision == SHAMPOO_PRECISION_AUTO && !(prm->kappa32 >= 1.f))
    return fail(h, SHAMPOO_EINVAL, "kappa32 must be >= 1");
  for (int j = 0; j < njobs; ++j) {
    if (jobs[j].n < 1 || jobs[j].n > kMaxDim)
      return fail(h, SHAMPOO_EINVAL, "job %d: n = %d outside [1, %d]", j, jobs[j].n, kMaxDim);
    if (!jobs[j].A || !jobs[j].X) return fail(h, SHAMPOO_EINVAL, "job %d: A or X is NULL", j);
    if (jobs[j].A == jobs[j].X) return fail(h, SHAMPOO_EINVAL, "job %d: A and X alias", j);
  }
  const int prec = prm->precision;
  const RootLayout L = root_layout(jobs, njobs, prec);
  if (ws_bytes < L.total)
    return fail(h, SHAMPOO_ENOMEM, "workspace %zu bytes < %zu needed", ws_bytes, L.total);
  DeviceGuard g(h->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  RootState* st = reinterpret_cast<RootState*>(ws + L.state);
  int* dcount = reinterpret_cast<int*>(ws + L.counts);
  int up = 0, full = 0, flat = 0;
  const NewtonJob<float>* j32 = nullptr;
  const NewtonJob<double>* j64 = nullptr;
  if (prec != SHAMPOO_PRECISION_FP64) {
    auto t = newton_table<float>(jobs, njobs, ws, L, &up, &full, &flat);
    const void* d = nullptr;
    STATUS_TRY(upload_table(h, t.data(), t.size() * sizeof(t[0]), s, &d));
    j32 = static_cast<const NewtonJob<float>*>(d);
  }
  if (prec != SHAMPOO_PRECISION_FP32) {
    auto t = newton_table<double>(jobs, njobs, ws, L, &up, &full, &flat);
    const void* d = nullptr;
    STATUS_TRY(upload_table(h, t.data(), t.size() * sizeof(t[0]), s, &d));
    j64 = static_cast<const NewtonJob<double>*>(d);
  }
  // upper-tile map of the product launches: logical tile -> (job, ti, tj)
  TileLists tl{};
  {
    std::vector<uint32_t> tm;
    std::vector<int> ub;
    tm.reserve(up);
    ub.reserve(njobs + 1);
    int ndiag = 0;
    for (int j = 0; j < njobs; ++j) {
      ub.push_back((int)tm.size());
      const int T = cdiv(jobs[j].n, kTile);
      for (int ti = 0; ti < T; ++ti)
        for (int tj = ti; tj < T; ++tj) tm.push_back(pack_tile(j, ti, tj));
      ndiag += T;
    }
    ub.push_back((int)tm.size());
    const void* d = nullptr;
    STATUS_TRY(upload_table(h, tm.data(), tm.size() * sizeof(uint32_t), s, &d));
    tl.tmap = static_cast<const uint32_t*>(d);
    STATUS_TRY(upload_table(h, ub.data(), ub.size() * sizeof(int), s, &d));
    tl.ubegin = static_cast<const int*>(d);
    tl.tlist = reinterpret_cast<uint32_t*>(ws + L.tlist);
    tl.tcount = reinterpret_cast<int*>(ws + L.tcount);
    for (int j = 1; j < njobs; ++j) tl.mixed |= jobs[j].n != jobs[0].n;
    tl.diag_last = !tl.mixed && ndiag <= 8 * kDiagLastMaxPerXcd;
  }
  // full-grid tiles of the warm start's general products
  TileLists tf{};
  if (warm) {
    std::vector<uint32_t> tm;
    std::vector<int> fb;
    tm.reserve(full);
    fb.reserve(njobs + 1);
    for (int j = 0; j < njobs; ++j) {
      fb.push_back((int)tm.size());
      const int T = cdiv(jobs[j].n, kTile);
      for (int ti = 0; ti < T; ++ti)
        for (int tj = 0; tj < T; ++tj) tm.push_back(pack_tile(j, ti, tj));
    }
    fb.push_back((int)tm.size());
    const void* d = nullptr;
    STATUS_TRY(upload_table(h, tm.data(), tm.size() * sizeof(uint32_t), s, &d));
    tf.tmap = static_cast<const uint32_t*>(d);
    STATUS_TRY(upload_table(h, fb.data(), fb.size() * sizeof(int), s, &d));
    tf.ubegin = static_cast<const int*>(d);
    tf.tlist = reinterpret_cast<uint32_t*>(ws + L.tlistf);
    tf.tcount = reinterpret_cast<int*>(ws + L.tcountf);
    tf.mixed = tl.mixed;
  }
  const int nb1 = cdiv(njobs, 64);
  const int tail_all = prec == SHAMPOO_PRECISION_FP64 ? 1 : 0;
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
    hipLaunchKernelGGL(root_reset_kernel, dim3(nb1), dim3(64), 0, s, st, njobs, 0, tail_all ? 64 : 32);
  }));
  // Prologue, shared by both precisions: MaxSV, Frobenius partials, z.
  const double eps = (double)prm->eps;
  if (prm->eps_relative) {
    // MaxSV: a tile pass and a reduce pass per power step over all
    // matrices; matrices whose estimate has settled skip the rest.
    STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
      if (j32)
        hipLaunchKernelGGL(maxsv_init_kernel<float>, dim3(njobs), dim3(kThreads), 0, s, j32, njobs, st);
      else
        hipLaunchKernelGGL(maxsv_init_kernel<double>, dim3(njobs), dim3(kThreads), 0, s, j64, njobs, st);
    }));
    const double mtol = (double)prm->maxsv_tol;
    for (int k = 0; k < prm->maxsv_steps; ++k) {
      const int last = k + 1 == prm->maxsv_steps;
      STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
        if (j32) {
          hipLaunchKernelGGL(maxsv_step_kernel<float>, dim3(full), dim3(kThreads), 0, s, j32, njobs,
                             (const RootState*)st, full, 0);
          hipLaunchKernelGGL(maxsv_reduce_kernel<float>, dim3(njobs), dim3(kSvThreads), 0, s, j32, njobs, st, mtol,
                             eps, last);
        } else {
          hipLaunchKernelGGL(maxsv_step_kernel<double>, dim3(full), dim3(kThreads), 0, s, j64, njobs,
                             (const RootState*)st, full, 0);
          hipLaunchKernelGGL(maxsv_reduce_kernel<double>, dim3(njobs), dim3(kSvThreads), 0, s, j64, njobs, st, mtol,
                             eps, last);
        }
      }));
    }
  }
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
    if (j32) {
      hipLaunchKernelGGL(frob_kernel<float>, dim3(up), dim3(kThreads), 0, s, j32, njobs, st, up);
      hipLaunchKernelGGL(root_prep_kernel<float>, dim3(nb1), dim3(64), 0, s, j32, njobs, st, p, prm->eps_relative, eps);
    } else {
      hipLaunchKernelGGL(frob_kernel<double>, dim3(up), dim3(kThreads), 0, s, j64, njobs, st, up);
      hipLaunchKernelGGL(root_prep_kernel<double>, dim3(nb1), dim3(64), 0, s, j64, njobs, st, p, prm->eps_relative,
                         eps);
    }
  }));
  // AUTO: the fp32 phase's cap, from the scalar recurrence for the
  // smallest scaled eigenvalue (p + 1) / (2 kappa32), and m1, the smallest
  // scaled eigenvalue that still converges within it
  int cap32 = prm->max_iters;
  double m1 = 0.0;
  if (prec == SHAMPOO_PRECISION_AUTO) {
    const double tl = std::max((double)prm->tol, 1e-6);
    const double m0 = std::min(1.0, (p + 1.0) / (2.0 * (double)prm->kappa32));
    const int k32 = host_scalar_iters(m0, p, tl, 1000) + 1;
    cap32 = std::min(cap32, std::max(k32, 1));
    double lo = 1e-300, hi = 1.0;
    for (int b = 0; b < 200; ++b) {
      const double mid = sqrt(lo * hi);
      if (host_scalar_iters(mid, p, tl, cap32 + 1) <= cap32) hi = mid; else lo = mid;
    }
    m1 = hi;
  }
  // AUTO with scaled damping (MaxSV ran): the Lanczos condition witness
  // sends matrices that the fp32 cap would certainly reject straight to fp64
  if (prec == SHAMPOO_PRECISION_AUTO && prm->eps_relative && !warm && j32) {
    STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
      hipLaunchKernelGGL(lanczos_init_kernel<float>, dim3(njobs), dim3(kThreads), 0, s, j32, njobs, st);
    }));
    for (int k = 0; k < kLanczosMax; ++k) {
      STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
        hipLaunchKernelGGL(maxsv_step_kernel<float>, dim3(full), dim3(kThreads), 0, s, j32, njobs,
                           (const RootState*)st, full, 1);
        hipLaunchKernelGGL(lanczos_reduce_kernel<float>, dim3(njobs), dim3(kSvThreads), 0, s, j32, njobs, st, p, m1,
                           kLanczosMax);
      }));
    }
  }
  // warm phase; -1: unknown number of matrices handed to the cold start
  int warm_aborts = -1;
  if (warm) {
    if (j32)
      STATUS_TRY(warm_phase<float>(h, j32, tf, njobs, st, dcount, full, prog, p, prm->tol, comm_tol, prm->max_iters,
                                   prm->poll, SHAMPOO_KCLASS_NEWTON_WARM, warm_out, s, &warm_aborts));
    else
      STATUS_TRY(warm_phase<double>(h, j64, tf, njobs, st, dcount, full, prog, p, prm->tol, comm_tol,
                                    prm->max_iters, prm->poll, SHAMPOO_KCLASS_NEWTON_WARM, warm_out, s, &warm_aborts));
  }
  if (tail_all) {
    // every matrix (after a warm phase: every matrix it handed on) goes to
    // the fp64 phase
    STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
      hipLaunchKernelGGL(root_escalate_kernel, dim3(1), dim3(kThreads), 0, s, st, njobs, dcount + 2 * kCountRing + 2);
      if (warm)  // results the warm phase accepted
        hipLaunchKernelGGL(root_output_kernel<double>, dim3(flat), dim3(kThreads), 0, s, j64, njobs, st, flat, 0, p);
    }));
  }
  int run64 = tail_all && !(warm && warm_aborts == 0);
  if (j32) {
    const int cap = cap32;
    const float* esc = nullptr;
    int esc_n = 0;
    if (prec == SHAMPOO_PRECISION_AUTO) {
      // Early escalation: m1 is the smallest scaled eigenvalue that still
      // converges within the cap; after k iterations it has reached f^k(m1)
      // (f(m) = ((p+1-m)/p)^p m), so a residual above 1 - f^k(m1) means the
      // matrix would reach the cap unconverged.
      std::vector<float> thr(cap);
      double m = m1;
      for (int k = 0; k < cap; ++k) {
        m = pow((p + 1.0 - m) / p, p) * m;
        thr[k] = (float)(1.0 - m);  // escalating a borderline matrix early is harmless
      }
      const void* d = nullptr;
      STATUS_TRY(upload_table(h, thr.data(), thr.size() * sizeof(float), s, &d));
      esc = static_cast<const float*>(d);
      esc_n = cap;
    }
    int fails = -1;
    if (warm && warm_aborts == 0)
      fails = 0;  // every warm result was accepted: no cold start
    else
      STATUS_TRY(newton_phase<float>(h, j32, tl, njobs, st, dcount, up, full, flat, prog, p, prm->scaling, prm->tol,
                                     cap, prm->poll, SHAMPOO_KCLASS_NEWTON_F32, esc, esc_n, s, &fails));
    if (prec == SHAMPOO_PRECISION_AUTO) {
      int* esc_count = dcount + 2 * kCountRing + 2;
      STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
        hipLaunchKernelGGL(root_escalate_kernel, dim3(1), dim3(kThreads), 0, s, st, njobs, esc_count);
      }));
      if (!prm->poll) {
        run64 = 1;
      } else if (fails >= 0) {
        run64 = fails > 0;  // known from the last poll: no synchronisation
      } else {
        // the phase ended at its cap with matrices still running
        HIP_TRY(h, hipMemcpyAsync(h->pinned + 2 * kCountRing + 2, esc_count, sizeof(int), hipMemcpyDeviceToHost, s));
        HIP_TRY(h, hipStreamSynchronize(s));
        run64 = h->pinned[2 * kCountRing + 2] > 0;
      }
    }
    STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
      hipLaunchKernelGGL(root_output_kernel<float>, dim3(flat), dim3(kThreads), 0, s, j32, njobs, st, flat, 0, p);
    }));
  }
  if (run64) {
    if (!tail_all) {
      STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
        hipLaunchKernelGGL(root_reset_kernel, dim3(nb1), dim3(64), 0, s, st, njobs, 1, 64);
      }));
    }
    STATUS_TRY(newton_phase<double>(h, j64, tl, njobs, st, dcount, up, full, flat, prog, p, prm->scaling, prm->tol,
                                    prm->max_iters, prm->poll, SHAMPOO_KCLASS_NEWTON_F64, nullptr, 0, s));
    STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
      hipLaunchKernelGGL(root_output_kernel<double>, dim3(flat), dim3(kThreads), 0, s, j64, njobs, st, flat, 1, p);
    }));
  }
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_ROOT_AUX, s, [&] {
    if (j32)
      hipLaunchKernelGGL(root_info_kernel<float>, dim3(nb1), dim3(64), 0, s, j32, njobs, st, p, prm->tol, (void*)info);
    else
      hipLaunchKernelGGL(root_info_kernel<double>, dim3(nb1), dim3(64), 0, s, j64, njobs, st, p, prm->tol, (void*)info);
  }));
  return tables_done(h, s);
}
}  // namespace

extern "C" {

shampoo_status shampoo_inv_root_batched(void* handle, const shampoo_root_job* jobs, int njobs,
                                        const shampoo_root_params* prm, void* workspace, size_t ws_bytes,
                                        shampoo_root_info* info, void* stream) {
  return inv_root_impl(static_cast<Handle*>(handle), jobs, njobs, prm, 0, 0.f, workspace, ws_bytes, info, nullptr,
                       stream);
}

shampoo_status shampoo_inv_root_warm_batched(void* handle, const shampoo_root_job* jobs, int njobs,
                                             const shampoo_root_params* prm, float comm_tol, void* workspace,
                                             size_t ws_bytes, shampoo_root_info* info, int32_t* warm_out,
                                             void* stream) {
  return inv_root_impl(static_cast<Handle*>(handle), jobs, njobs, prm, 1, comm_tol, workspace, ws_bytes, info,
                       warm_out, stream);
}

shampoo_status shampoo_timing_enable(void* handle, int enable) {
  Handle* h = static_cast<Handle*>(handle);
  if (!h) return SHAMPOO_EINVAL;
  h->timing = enable != 0;
  return SHAMPOO_OK;
}

shampoo_status shampoo_timing_read(void* handle, int kclass, double* total_ms, int64_t* launches) {
  Handle* h = static_cast<Handle*>(handle);
  if (!h) return SHAMPOO_EINVAL;
  if (kclass < 0 || kclass >= SHAMPOO_KCLASS_COUNT) return fail(h, SHAMPOO_EINVAL, "bad kernel class %d", kclass);
  DeviceGuard g(h->device);
  double ms = 0.0;
  int64_t n = 0;
  std::vector<TimedLaunch> keep;
  for (auto& t : h->timed) {
    if (t.cls != kclass) {
      keep.push_back(t);
      continue;
    }
    HIP_TRY(h, hipEventSynchronize(t.b));
    float x = 0.f;
    HIP_TRY(h, hipEventElapsedTime(&x, t.a, t.b));
    ms += x;
    ++n;
    h->spare_events.push_back(t.a);
    h->spare_events.push_back(t.b);
  }
  h->timed.swap(keep);
  if (total_ms) *total_ms = ms;
  if (launches) *launches = n;
  return SHAMPOO_OK;
}


// ---------------------------------------------------------------- embeddings
size_t shampoo_embedding_workspace_bytes(int nnz, int dim) {
  if (nnz < 1 || nnz > kMaxEmbEntries || dim < 1 || dim > kMaxDim) return 0;
  return emb_layout(nnz, dim).total;
}

shampoo_status shampoo_embedding_rows(void* handle, const int32_t* idx, const int32_t* feat, const float* weight,
                                      int nnz, int64_t vocab, const float* dy, int m, int dim, int64_t ld_dy,
                                      int32_t* rows, float* U, int32_t* count, void* workspace, size_t ws_bytes,
                                      void* stream) {
  Handle* h = static_cast<Handle*>(handle);
  if (!h) return SHAMPOO_EINVAL;
  h->err.clear();
  STATUS_TRY(emb_check(h, nnz, dim));
  if (vocab < 1 || vocab >= INT32_MAX) return fail(h, SHAMPOO_EINVAL, "vocab = %lld outside [1, 2^31 - 1)", (long long)vocab);
  if (m < 1) return fail(h, SHAMPOO_EINVAL, "m = %d < 1", m);
  if (ld_dy < dim) return fail(h, SHAMPOO_EINVAL, "ld_dy %lld < dim %d", (long long)ld_dy, dim);
  if (!idx || !dy || !rows || !U || !count || !workspace)
    return fail(h, SHAMPOO_EINVAL, "idx, dy, rows, U, count or workspace is NULL");
  const EmbLayout L = emb_layout(nnz, dim);
  if (ws_bytes < L.total) return fail(h, SHAMPOO_ENOMEM, "workspace %zu bytes < %zu needed", ws_bytes, L.total);
  DeviceGuard g(h->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  int32_t* keys = reinterpret_cast<int32_t*>(ws + L.keys);
  int32_t* vals = reinterpret_cast<int32_t*>(ws + L.vals);
  int32_t* keys_s = reinterpret_cast<int32_t*>(ws + L.keys_s);
  int32_t* vals_s = reinterpret_cast<int32_t*>(ws + L.vals_s);
  int32_t* uniq = reinterpret_cast<int32_t*>(ws + L.uniq);
  int32_t* lens = reinterpret_cast<int32_t*>(ws + L.lens);
  int32_t* offs = reinterpret_cast<int32_t*>(ws + L.offs);
  int32_t* nruns = reinterpret_cast<int32_t*>(ws + L.nruns);
  float* cpart = reinterpret_cast<float*>(ws + L.cpart);
  const int32_t v32 = (int32_t)vocab;
  int bits = 1;
  while (bits < 31 && (int64_t(1) << bits) <= vocab) ++bits;  // keys lie in [0, vocab]
  // rocPRIM temporary storage (sized by a query; grown on the handle)
  size_t t_sort = 0, t_rle = 0, t_scan = 0;
  HIP_TRY(h, rocprim::radix_sort_pairs(nullptr, t_sort, keys, keys_s, vals, vals_s, (unsigned)nnz, 0, bits, s));
  HIP_TRY(h, rocprim::run_length_encode(nullptr, t_rle, keys_s, (unsigned)nnz, uniq, lens, nruns, s));
  HIP_TRY(h, rocprim::exclusive_scan(nullptr, t_scan, lens, offs, 0, (unsigned)nnz, rocprim::plus<int32_t>(), s));
  size_t tb = std::max(t_sort, std::max(t_rle, t_scan));
  STATUS_TRY(grow(h, &h->sort_tmp, &h->sort_tmp_cap, std::max<size_t>(tb, 256), s));
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_EMB, s, [&] {
    hipLaunchKernelGGL(emb_keys_kernel, dim3(cdiv(nnz, kThreads)), dim3(kThreads), 0, s, idx, feat, nnz, v32, m,
                       keys, vals, lens);
  }));
  // stable sort by row (entries of a row keep their order), runs, run offsets
  hipError_t re = hipSuccess;
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_EMB, s, [&] {
    size_t t = h->sort_tmp_cap;
    re = rocprim::radix_sort_pairs(h->sort_tmp, t, keys, keys_s, vals, vals_s, (unsigned)nnz, 0, bits, s);
  }));
  HIP_TRY(h, re);
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_EMB, s, [&] {
    size_t t = h->sort_tmp_cap;
    re = rocprim::run_length_encode(h->sort_tmp, t, keys_s, (unsigned)nnz, uniq, lens, nruns, s);
  }));
  HIP_TRY(h, re);
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_EMB, s, [&] {
    size_t t = h->sort_tmp_cap;
    re = rocprim::exclusive_scan(h->sort_tmp, t, lens, offs, 0, (unsigned)nnz, rocprim::plus<int32_t>(), s);
  }));
  HIP_TRY(h, re);
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_EMB, s, [&] {
    hipLaunchKernelGGL(emb_chunk_kernel, dim3(cdiv(nnz, kEmbChunk)), dim3(kThreads), 0, s, uniq, lens, offs, nruns,
                       vals_s, feat, weight, dy, ld_dy, dim, v32, nnz, U, cpart);
  }));
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_EMB, s, [&] {
    hipLaunchKernelGGL(emb_fix_kernel, dim3(nnz), dim3(kThreads), 0, s, uniq, lens, offs, nruns, dim, v32, nnz,
                       (const float*)cpart, rows, U, count);
  }));
  return SHAMPOO_OK;
}

shampoo_status shampoo_embedding_stats(void* handle, const float* U, const int32_t* count, int nnz, int dim,
                                       float* R, float beta2, void* workspace, size_t ws_bytes, void* stream) {
  Handle* h = static_cast<Handle*>(handle);
  if (!h) return SHAMPOO_EINVAL;
  h->err.clear();
  STATUS_TRY(emb_check(h, nnz, dim));
  if (!U || !count || !R) return fail(h, SHAMPOO_EINVAL, "U, count or R is NULL");
  if (!(beta2 > 0.f && beta2 <= 1.f)) return fail(h, SHAMPOO_EINVAL, "beta2 %g outside (0, 1]", (double)beta2);
  const EmbLayout L = emb_layout(nnz, dim);
  if (L.splits > 1 && (!workspace || ws_bytes < L.total))
    return fail(h, SHAMPOO_ENOMEM, "workspace %zu bytes < %zu needed", ws_bytes, L.total);
  DeviceGuard g(h->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const float c = beta2 == 1.0f ? 1.0f : 1.0f - beta2;
  const bool al = aligned16(U) && (dim % 4) == 0;
  const size_t pstride = align256((size_t)dim * dim * sizeof(float)) / sizeof(float);
  float* part = L.splits > 1 ? reinterpret_cast<float*>(static_cast<char*>(workspace) + L.part) : nullptr;
  std::vector<GemmProblem> probs;
  for (int q = 0; q < L.splits; ++q) {
    GemmProblem p{};
    p.A = U; p.B = U;
    p.lda = p.ldb = dim;
    p.a_rows = p.b_rows = nnz; p.a_cols = p.b_cols = dim;
    p.M = p.N = dim; p.K = nnz;
    p.sym = 1;
    p.a_aligned = p.b_aligned = al;
    p.kcount = count; p.koff = q; p.ksplit = L.splits;  // split q of the active rows
    if (part) {
      p.C = part + (size_t)q * pstride; p.ldc = dim; p.alpha = 1.f; p.beta = 0.f;
    } else {
      p.C = R; p.ldc = dim; p.alpha = c; p.beta = beta2;
    }
    probs.push_back(p);
  }
  // R = U^T U: both operands read row by row of U (k = row of U).
  STATUS_TRY((run_gemm<float, kLayoutK, float, kLayoutK, true>(h, probs, s, SHAMPOO_KCLASS_STATS)));
  if (part) {
    const int64_t n = (int64_t)dim * dim;
    STATUS_TRY(launch(h, SHAMPOO_KCLASS_STATS, s, [&] {
      hipLaunchKernelGGL(emb_reduce_kernel, dim3((unsigned)cdiv((int)cdiv(n, 4), kThreads)), dim3(kThreads), 0, s,
                         (const float*)part, L.splits, (int64_t)pstride, n, c, beta2, R);
    }));
  }
  return tables_done(h, s);
}

shampoo_status shampoo_embedding_precondition(void* handle, const float* U, const int32_t* count, int nnz, int dim,
                                              const float* Rr, float* P, void* stream) {
  Handle* h = static_cast<Handle*>(handle);
  if (!h) return SHAMPOO_EINVAL;
  h->err.clear();
  STATUS_TRY(emb_check(h, nnz, dim));
  if (!U || !count || !Rr || !P) return fail(h, SHAMPOO_EINVAL, "U, count, Rr or P is NULL");
  DeviceGuard g(h->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  std::vector<GemmProblem> probs(1);
  GemmProblem& p = probs[0];
  p = GemmProblem{};
  p.A = U; p.lda = dim; p.a_rows = nnz; p.a_cols = dim; p.a_aligned = aligned16(U) && (dim % 4) == 0;
  p.B = Rr; p.ldb = dim; p.b_rows = dim; p.b_cols = dim; p.b_aligned = aligned16(Rr) && (dim % 4) == 0;
  p.C = P; p.ldc = dim; p.M = nnz; p.N = dim; p.K = dim;
  p.alpha = 1.f; p.beta = 0.f;
  p.mcount = count;
  STATUS_TRY((run_gemm<float, kLayoutRow, float, kLayoutK, true>(h, probs, s, SHAMPOO_KCLASS_PRECOND)));
  return tables_done(h, s);
}

shampoo_status shampoo_embedding_graft(void* handle, const int32_t* rows, const int32_t* count, int nnz, int dim,
                                       const float* U, const float* P, float* W, float* D, int64_t vocab,
                                       int64_t ldw, float eta0, int use_shampoo, float* norms, void* stream) {
  Handle* h = static_cast<Handle*>(handle);
  if (!h) return SHAMPOO_EINVAL;
  h->err.clear();
  STATUS_TRY(emb_check(h, nnz, dim));
  if (vocab < 1 || vocab >= INT32_MAX) return fail(h, SHAMPOO_EINVAL, "vocab = %lld outside [1, 2^31 - 1)", (long long)vocab);
  if (ldw < dim) return fail(h, SHAMPOO_EINVAL, "ldw %lld < dim %d", (long long)ldw, dim);
  if (!rows || !count || !U || !W || !D || (use_shampoo && !P))
    return fail(h, SHAMPOO_EINVAL, "rows, count, U, W, D or P is NULL");
  if (!isfinite(eta0)) return fail(h, SHAMPOO_EINVAL, "eta0 is not finite");
  DeviceGuard g(h->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  GraftBlock b{};
  b.G = U; b.P = use_shampoo ? P : nullptr; b.W = W; b.D = D; b.Mg = nullptr; b.Ps = nullptr;
  b.ld = dim; b.rows = nnz; b.cols = dim;
  b.wrows = rows; b.count = count; b.ldw = ldw; b.wlimit = vocab;
  b.rows_per_chunk = std::max(1, 16384 / dim);
  b.nchunks = cdiv(nnz, b.rows_per_chunk);
  b.chunk_begin = 0;
  b.part_begin = 0;
  b.nparts = b.nchunks;
  b.vec4 = (dim % 4) == 0 && (ldw % 4) == 0 && aligned16(U) && aligned16(W) && aligned16(D) &&
           (!b.P || aligned16(b.P));
  const int total = b.nchunks;
  const void* d = nullptr;
  STATUS_TRY(upload_table(h, &b, sizeof(b), s, &d));
  STATUS_TRY(grow(h, &h->partial, &h->partial_cap, (size_t)total * 2 * sizeof(double), s));
  double* part = static_cast<double*>(h->partial);
  const GraftBlock* db = static_cast<const GraftBlock*>(d);
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_GRAFT, s, [&] {
    hipLaunchKernelGGL((graft_pass1_kernel<float, false>), dim3(total), dim3(kThreads), 0, s, db, 1, total, 0.f, use_shampoo,
                       part);
  }));
  STATUS_TRY(launch(h, SHAMPOO_KCLASS_GRAFT, s, [&] {
    hipLaunchKernelGGL((graft_pass2_kernel<float, false>), dim3(total), dim3(kThreads), 0, s, db, 1, total, eta0, 0.f,
                       use_shampoo, (const double*)part, norms);
  }));
  return tables_done(h, s);
}

}  // extern "C"
