// Device code of the Oscars hot path for gfx950 (CDNA4).
//
//  * gemm_kernel   grouped MFMA GEMM, one launch per layer and pass, grid z =
//                  active replica slot.  Three pass shapes share one body:
//                  forward (NT), backward-data (NN), backward-weight (TN) with
//                  the SGD update x <- x - eta g(x) of Eq. 4 fused into the
//                  epilogue, so weight gradients never reach HBM.
//  * softmax_ce    logit gradient of the mean softmax cross-entropy.
//  * cast_bf16     fp32 master -> bf16 working copy (bf16 models).
//  * aggregate     the parameter server's average of Eq. 4 as a pairwise-tree
//                  K-way reduction, 128-bit loads, lane groups combined with
//                  cross-lane shuffles, optional broadcast back to every replica.
//
// Tiles: 128 x 128 outputs per workgroup; the wave layout depends on the pass
// (see Shape below).  LDS holds both operands K-contiguous:
// 128 rows x 128 bytes (64 bf16 or 32 fp32), 16-byte chunks placed at
// chunk ^ ((row ^ row >> 3) & 7) so that MFMA operand reads (consecutive rows,
// one chunk) and transposing writes (rows 8 apart) both spread over the banks.
// Operands stored M/N-contiguous in memory (weights in backward-data, both
// operands of backward-weight) are transposed on their way into LDS.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <map>
#include <mutex>
#include <new>
#include <tuple>
#include <type_traits>
#include <vector>

#include "../../include/oscars.h"
#include "kernels.h"

namespace oscars {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// Workgroup tile shapes.  All shapes use the same K tile (BK) and the same
// MFMA k-grouping, so an output element is summed in the same order whatever
// the shape: the shape only decides which workgroup computes it.
//   BM x BN outputs, WAVES_M x WAVES_N waves (each BM/WAVES_M x BN/WAVES_N),
//   ST register stages for the long-K passes, MINW minimum waves per SIMD.
template <int BM_, int BN_, int WM_, int WN_, int STAGES, int MINW>
struct Shape {
  static constexpr int BM = BM_, BN = BN_;
  static constexpr int WAVES_M = WM_, WAVES_N = WN_;
  static constexpr int NT = 64 * WM_ * WN_;          // threads
  static constexpr int MI = BM_ / (32 * WM_);        // MFMA blocks per wave along M
  static constexpr int NJ = BN_ / (32 * WN_);        // and along N
  static constexpr int ST = STAGES;
  static constexpr int MIN_WAVES = MINW;
};
// Forward / backward-data (K = layer width):
//   batches above 128: the whole batch in one tile, 128 x 256 with 8 waves
//   (W) or 64 x 256 with 4 waves (V), every wave 64 x 64, so each weight is
//   read once per launch and each LDS operand read feeds two MFMAs;
//   smaller batches: 128 x 128 with 8 waves (L), 64 x 128 (M) or 64 x 64 (S)
//   with 4 waves.  The largest tile that still gives every CU a workgroup is
//   taken; below that, the K chunks are split over workgroups (split-K).
// Backward-weight + update (K = batch): 128 x 128, 4 waves, one stage.
enum { SHAPE_L = 0, SHAPE_M = 1, SHAPE_S = 2, SHAPE_W = 3, SHAPE_V = 4 };
template <int MODE, int SID> struct ShapeOf;
template <int MODE> struct ShapeOf<MODE, SHAPE_L> { typedef Shape<128, 128, 2, 4, 2, 1> type; };
template <int MODE> struct ShapeOf<MODE, SHAPE_M> { typedef Shape<64, 128, 1, 4, 2, 1> type; };
template <int MODE> struct ShapeOf<MODE, SHAPE_S> { typedef Shape<64, 64, 2, 2, 2, 1> type; };
// W and V are bf16-only and stream both K tiles straight into LDS (ST = LDS
// stages, see gemm_dma_kernel).
template <int MODE> struct ShapeOf<MODE, SHAPE_W> { typedef Shape<128, 256, 2, 4, 3, 1> type; };
template <int MODE> struct ShapeOf<MODE, SHAPE_V> { typedef Shape<64, 256, 1, 4, 3, 1> type; };

// Forward and backward-data sum K in chunks of KCHUNK elements: each chunk
// from zero, in K order, and the chunk sums left to right,
// ((p0 + p1) + p2) + ...  The order does not depend on the tile shape or on
// whether the chunks of one output are summed in one workgroup (non-split)
// or written as partials by one workgroup each and summed by the reduce
// kernel (split-K), so a replica's result never depends on how many
// replicas share the launch.
constexpr int KCHUNK = GEMM_KCHUNK;
#ifndef WGRAD_MIN_WAVES
#define WGRAD_MIN_WAVES 3
#endif
#ifndef WGRAD_PRE
#define WGRAD_PRE 8
#endif
template <> struct ShapeOf<GEMM_WGRAD, SHAPE_L> { typedef Shape<128, 128, 2, 2, 1, 2> type; };

constexpr int ROW_U32 = 32;               // one LDS tile row: 128 bytes

__device__ __forceinline__ int lds_word(int row, int chunk) {
  return row * ROW_U32 + ((chunk ^ ((row ^ (row >> 3)) & 7)) << 2);
}

// A compile-time integer passed as an argument (static register indices).
template <int U> struct Ic { static constexpr int value = U; };

// fp32 -> bf16, round to nearest even on the fp32 bits.
__device__ __forceinline__ uint32_t f2bf(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

template <bool BF16> struct El;
template <> struct El<true> {
  typedef uint16_t T;
  static constexpr int CH = 8;   // elements per 16-byte chunk
  static constexpr int BK = 64;  // K per LDS tile
};
template <> struct El<false> {
  typedef float T;
  static constexpr int CH = 4;
  static constexpr int BK = 32;
};

// Loaders never branch and never depend on a load inside the K loop: row
// pointers (gathered or not) are set up once, before the loop; an
// out-of-range lane reads the operand's first chunk (always valid memory) and
// keeps zeros instead.  `ext` is the chunked extent of the contiguous
// dimension: a multiple of the chunk, with memory up to it readable (zero
// padding beyond the logical size where needed).
// Out-of-range lanes read these zeros instead of selecting zeros after the
// load, so nothing waits on a load before its data is stored to LDS.
__device__ __attribute__((aligned(16))) uint32_t k_zero16[4];

template <typename T>
__device__ __forceinline__ u32x4 load16(bool ok, const T* p) {
  return *reinterpret_cast<const u32x4*>(ok ? static_cast<const void*>(p)
                                            : static_cast<const void*>(k_zero16));
}

// Tile of an operand stored K-contiguous: 128 rows (M or N) x BK.
//   rows valid: row0 + r < R (row r of memory is gather[row0 + r] if gathered);
//   chunk valid: k < ext.
template <bool BF16, int NTHR, int ROWS>
struct RowSrc {
  typedef typename El<BF16>::T T;
  static_assert(ROWS * 8 % NTHR == 0, "whole chunks per thread");
  static constexpr int P = ROWS * 8 / NTHR;
  const T* rowp[P];
  bool rowok[P];
  __device__ __forceinline__ void init(const T* base, int64_t ld, const int32_t* gather, int row0,
                                       int R, int tid) {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int gr = row0 + ((tid + NTHR * p) >> 3);
      rowok[p] = gr < R;
      const int grc = gr < R ? gr : R - 1;
      const int64_t row = gather ? gather[grc] : grc;
      rowp[p] = base + row * ld;
    }
  }
};

template <bool BF16, int NTHR, int ROWS>
struct RowTile {
  typedef typename El<BF16>::T T;
  static constexpr int CH = El<BF16>::CH;
  static constexpr int P = ROWS * 8 / NTHR;
  u32x4 v[P];
  __device__ __forceinline__ void load(const RowSrc<BF16, NTHR, ROWS>& src, const T* base, int k0,
                                       int ext, int tid) {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int k = k0 + ((tid + NTHR * p) & 7) * CH;
      const bool ok = src.rowok[p] && k < ext;
      v[p] = load16(ok, src.rowp[p] + k);
    }
  }
  // Copy of the loaded chunks to dst (same row index, row stride ld_dst).
  __device__ __forceinline__ void copy_out(T* dst, int64_t ld_dst, int row0, int R, int k0,
                                           int ext, int tid) const {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int idx = tid + NTHR * p, gr = row0 + (idx >> 3), k = k0 + (idx & 7) * CH;
      if (gr < R && k < ext)
        *reinterpret_cast<u32x4*>(dst + static_cast<int64_t>(gr) * ld_dst + k) = v[p];
    }
  }
  __device__ __forceinline__ void store(uint32_t* lds, int tid) const {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int idx = tid + NTHR * p;
      *reinterpret_cast<u32x4*>(lds + lds_word(idx >> 3, idx & 7)) = v[p];
    }
  }
};

// Tile of an operand stored M/N-contiguous ([K][MN] in memory), transposed
// into the K-contiguous LDS layout.  bf16: pairs of k rows are packed into
// 32-bit words; fp32: single words.
//   rows valid: k < K;  chunk valid: mn < ext.
template <bool BF16, int NTHR, int ROWS> struct TransTile;

template <int NTHR, int ROWS>
struct TransTile<true, NTHR, ROWS> {
  static constexpr int MC = ROWS / 8;  // 16-byte chunks per k row
  static_assert(32 * MC % NTHR == 0, "whole items per thread");
  static constexpr int P = 32 * MC / NTHR;
  u32x4 lo[P], hi[P];
  __device__ __forceinline__ void load(const uint16_t* base, int64_t ld, int mn0, int ext, int k0,
                                       int K, int tid) {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int idx = tid + NTHR * p, mc = idx % MC, kp = idx / MC;
      const int k = k0 + 2 * kp, mn = mn0 + 8 * mc;
      const bool ok0 = k < K && mn < ext, ok1 = k + 1 < K && mn < ext;
      lo[p] = load16(ok0, base + k * ld + mn);
      hi[p] = load16(ok1, base + (k + 1) * ld + mn);
    }
  }
  // The loaded registers count as written here (an empty asm, ordered after
  // the preceding volatile asm): their uses stay below this point.
  __device__ __forceinline__ void pin() {
#pragma unroll
    for (int p = 0; p < P; ++p) asm volatile("" : "+v"(lo[p]), "+v"(hi[p]));
  }
  __device__ __forceinline__ void store(uint32_t* lds, int tid) const {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int idx = tid + NTHR * p, mc = idx % MC, kp = idx / MC;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t a = lo[p][e >> 1], b = hi[p][e >> 1];
        const uint32_t w = (e & 1) ? ((a >> 16) | (b & 0xFFFF0000u)) : ((a & 0xFFFFu) | (b << 16));
        lds[lds_word(8 * mc + e, kp >> 2) + (kp & 3)] = w;
      }
    }
  }
};

template <int NTHR, int ROWS>
struct TransTile<false, NTHR, ROWS> {
  static constexpr int MC = ROWS / 4;
  static_assert(32 * MC % NTHR == 0, "whole items per thread");
  static constexpr int P = 32 * MC / NTHR;
  u32x4 v[P];
  __device__ __forceinline__ void load(const float* base, int64_t ld, int mn0, int ext, int k0,
                                       int K, int tid) {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int idx = tid + NTHR * p, mc = idx % MC, kk = idx / MC;
      const int k = k0 + kk, mn = mn0 + 4 * mc;
      const bool ok = k < K && mn < ext;
      v[p] = load16(ok, base + k * ld + mn);
    }
  }
  __device__ __forceinline__ void store(uint32_t* lds, int tid) const {
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int idx = tid + NTHR * p, mc = idx % MC, kk = idx / MC;
#pragma unroll
      for (int e = 0; e < 4; ++e) lds[lds_word(4 * mc + e, kk >> 2) + (kk & 3)] = v[p][e];
    }
  }
};

// MI x NJ blocks of 32x32 MFMA of one wave over one LDS tile pair.  The
// wave's rows start at wm * 32 MI, its columns at wn * 32 NJ.  `after_reads(s)`
// runs once the operand reads of k group s are issued, before its MFMAs.
struct NoHook {
  __device__ __forceinline__ void operator()(int) const {}
};
template <bool BF16, int MI, int NJ, typename Hook = NoHook>
__device__ __forceinline__ void mma_tile(const uint32_t* As, const uint32_t* Bs, int wm, int wn,
                                         int lane, f32x16 (&acc)[MI][NJ],
                                         const Hook& after_reads = Hook()) {
  const int r = lane & 31, h = lane >> 5;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const int ch = 2 * s + h;
    u32x4 a[MI], b[NJ];
#pragma unroll
    for (int i = 0; i < MI; ++i)
      a[i] = *reinterpret_cast<const u32x4*>(As + lds_word(wm * 32 * MI + 32 * i + r, ch));
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      b[j] = *reinterpret_cast<const u32x4*>(Bs + lds_word(wn * 32 * NJ + 32 * j + r, ch));
    after_reads(s);
    if constexpr (BF16) {
      // lanes 0-31 hold k = 16s..16s+7 of their row, lanes 32-63 k = 16s+8..16s+15
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8, a[i]), __builtin_bit_cast(bf16x8, b[j]), acc[i][j], 0, 0, 0);
    } else {
      // lanes 0-31 hold k = 8s..8s+3, lanes 32-63 k = 8s+4..8s+7; MFMA t
      // contracts element t of every lane, i.e. k = 8s + t and 8s + 4 + t.
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
          for (int j = 0; j < NJ; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[i][t]),
                                                             __uint_as_float(b[j][t]), acc[i][j],
                                                             0, 0, 0);
    }
  }
}

// Flattened workgroup id L (the dispatch order: x fastest, then y) -> work
// item, such that the workgroups the hardware places on one XCD (L mod 8)
// take one contiguous range of the T work items.  The GEMM grids number
// their work slot-major, tile within slot: the tiles of one replica slot,
// which read the same activation (or delta) block, then share one XCD and
// its L2, and neighbouring tiles share their weight rows as well.
__device__ __forceinline__ int xcd_work(int L, int T) {
  const int x = L & 7, i = L >> 3, q = T >> 3, r = T & 7;
  return x < r ? x * (q + 1) + i : r * (q + 1) + (x - r) * q + i;
}

// Forward / backward-data output of four consecutive rows m..m+3 (cnt of them
// inside M) at column n of slot z: bias and ReLU (forward) or the ReLU mask of
// the layer below (backward-data), then bf16 or fp32 store.  epi_load reads
// what the epilogue needs (forward: the bias, 0 past cnt; backward-data: 1
// where the mask is positive, else 0), store_out_with applies it and stores.
template <bool BF16, int MODE>
__device__ __forceinline__ f32x4 epi_load(const GemmArgs& g, int z, int n, int m, int cnt,
                                          const float* master_in) {
  // One vector load, no branch (a branch around it would make the compiler
  // wait for it on the spot): the bias segment and the mask rows (the
  // activations of a layer l >= 1) are padded to 64 elements, so the four
  // elements from m (a multiple of 4 below M) are in range and aligned;
  // those past cnt are dropped.
  f32x4 a;
  if constexpr (MODE == GEMM_FWD) {
    const f32x4 b = *reinterpret_cast<const f32x4*>(master_in + g.b_off + m);
    for (int e = 0; e < 4; ++e) a[e] = e < cnt ? b[e] : 0.0f;
  } else {
    const int64_t am = z * g.mask_slot + static_cast<int64_t>(n) * g.mask_ld + m;
    bool pos[4];
    if constexpr (BF16) {
      const uint2 q = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(g.mask) + am);
      const uint32_t w[4] = {q.x & 0xFFFFu, q.x >> 16, q.y & 0xFFFFu, q.y >> 16};
      for (int e = 0; e < 4; ++e) pos[e] = w[e] != 0 && (w[e] & 0x8000u) == 0;
    } else {
      const f32x4 q = *reinterpret_cast<const f32x4*>(static_cast<const float*>(g.mask) + am);
      for (int e = 0; e < 4; ++e) pos[e] = q[e] > 0.0f;
    }
    for (int e = 0; e < 4; ++e) a[e] = e < cnt && pos[e] ? 1.0f : 0.0f;
  }
  return a;
}

template <bool BF16, int MODE>
__device__ __forceinline__ void store_out_with(const GemmArgs& g, int z, int n, int m, int cnt,
                                               f32x4 v, f32x4 a) {
  if constexpr (MODE == GEMM_FWD) {
    // out[b = n][o = m..m+3]
    for (int e = 0; e < 4; ++e) {
      float o = v[e] + a[e];
      v[e] = g.relu ? fmaxf(o, 0.0f) : o;
    }
  } else {
    for (int e = 0; e < 4; ++e) v[e] = a[e] != 0.0f ? v[e] : 0.0f;
  }
  const int64_t at = z * g.out_slot + static_cast<int64_t>(n) * g.out_ld + m;
  if (g.out_bf16) {
    uint16_t* o = static_cast<uint16_t*>(g.out) + at;
    if (cnt == 4) {
      uint2 pk;
      pk.x = f2bf(v[0]) | (f2bf(v[1]) << 16);
      pk.y = f2bf(v[2]) | (f2bf(v[3]) << 16);
      *reinterpret_cast<uint2*>(o) = pk;
    } else {
      for (int e = 0; e < cnt; ++e) o[e] = static_cast<uint16_t>(f2bf(v[e]));
    }
  } else {
    float* o = static_cast<float*>(g.out) + at;
    if (cnt == 4) {
      *reinterpret_cast<f32x4*>(o) = v;
    } else {
      for (int e = 0; e < cnt; ++e) o[e] = v[e];
    }
  }
}


// SPLIT: grid x = tiles x K chunks; the workgroup of (tile, chunk c) sums
// chunk c only and stores it as fp32 partial c of its outputs (g.part);
// splitk_reduce_kernel then sums the partials in chunk order and applies the
// epilogue.
template <bool BF16, int MODE, bool GATHER, int SID, bool SPLIT>
__global__ __launch_bounds__((ShapeOf<MODE, SID>::type::NT), (ShapeOf<MODE, SID>::type::MIN_WAVES)) void
gemm_kernel(GemmArgs g) {
  typedef typename El<BF16>::T T;
  typedef typename ShapeOf<MODE, SID>::type S;
  constexpr int NTHR = S::NT, WAVES_N = S::WAVES_N, MI = S::MI, NJ = S::NJ;
  constexpr int BM = S::BM, BN = S::BN;
  constexpr int BK = El<BF16>::BK;
  constexpr bool CHUNKED = MODE != GEMM_WGRAD;  // the batch (K of WGRAD) is one chunk
  static_assert(!SPLIT || CHUNKED, "split-K is for forward / backward-data");
  static_assert(KCHUNK % BK == 0, "whole K tiles per chunk");
  constexpr int TPC = KCHUNK / BK;  // K tiles per chunk
  // LDS: A tiles (BM rows) for buffers 0 and 1, then B tiles (BN rows).
  __shared__ __attribute__((aligned(16))) uint32_t lds_all[2 * (BM + BN) * ROW_U32];
  auto lds_a = [&](int buf) { return lds_all + buf * BM * ROW_U32; };
  auto lds_b = [&](int buf) { return lds_all + 2 * BM * ROW_U32 + buf * BN * ROW_U32; };

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N, h = lane >> 5;
  const int work = xcd_work(blockIdx.y * gridDim.x + blockIdx.x, gridDim.x * gridDim.y);
  const int z = work / gridDim.x;
  const int rep = g.order[z];
  const int M = g.M, N = g.N, K = g.K;
  const int gn = (N + BN - 1) / BN;
  const int t = work % gridDim.x;
  // Split: t = chunk * tiles + tile, so the workgroups of one XCD share the
  // B operand chunk (the batch's activations or deltas of that K range).
  const int nchunks = (K + KCHUNK - 1) / KCHUNK;
  const int tiles = SPLIT ? static_cast<int>(gridDim.x) / nchunks : static_cast<int>(gridDim.x);
  const int chunk = SPLIT ? t / tiles : 0, tile = SPLIT ? t % tiles : t;
  const int m0 = (tile / gn) * BM, n0 = (tile % gn) * BN;
  const int kbeg = SPLIT ? chunk * KCHUNK : 0;
  const int kend = SPLIT ? (K - kbeg < KCHUNK ? K : kbeg + KCHUNK) : K;

  const T* A = static_cast<const T*>(g.a) + (g.a_by_order ? rep : z) * g.a_slot;
  const T* B = static_cast<const T*>(g.b) + z * g.b_slot;
  float* master = g.master + static_cast<int64_t>(rep) * g.master_slot;
  const float* master_in = g.master_in + static_cast<int64_t>(rep) * g.master_in_slot;

  // A: weights K-contiguous in FWD, weights M-contiguous in DGRAD, activations
  // M-contiguous in WGRAD.  B: activations / delta K-contiguous in FWD and
  // DGRAD, delta N-contiguous in WGRAD.
  typename std::conditional<MODE == GEMM_FWD, RowTile<BF16, NTHR, BM>, TransTile<BF16, NTHR, BM>>::type ta;
  typename std::conditional<MODE == GEMM_WGRAD, TransTile<BF16, NTHR, BN>, RowTile<BF16, NTHR, BN>>::type tb;
  // Row pointers of the K-contiguous operands, fixed for the whole K loop.
  RowSrc<BF16, NTHR, BM> sa;
  RowSrc<BF16, NTHR, BN> sb;
  if constexpr (MODE == GEMM_FWD) sa.init(A, g.a_ld, nullptr, m0, M, tid);
  if constexpr (MODE != GEMM_WGRAD)
    sb.init(B, g.b_ld, GATHER ? g.gather + z * g.gather_slot : nullptr, n0, N, tid);
  // Forward layer 1 also keeps the gathered batch rows, contiguous, for the
  // backward-weight pass of that layer: K tile kt of the rows is written by
  // the workgroup of M tile kt mod (number of M tiles), so the copy is spread
  // over all workgroups of the launch.
  T* rows_out = GATHER ? static_cast<T*>(g.rows_out) + z * g.rows_out_slot : nullptr;
  const int gm = (M + BM - 1) / BM, mt = m0 / BM;

  // Accumulator element (i, j, r) sits at row m = mrow(i, r>>2) + (r & 3),
  // column n = ncol(j): four consecutive rows per lane and group r>>2.
  auto mrow = [&](int i, int q) { return m0 + wm * 32 * MI + 32 * i + 8 * q + 4 * h; };
  auto ncol = [&](int j) { return n0 + wn * 32 * NJ + 32 * j + (lane & 31); };

  // WGRAD: the fp32 master tile W[n0..n0+127][m0..m0+127] is fetched before
  // the K loop, so its HBM latency overlaps the products.  Layout: chunk
  // c = tid + NTHR p covers row n0 + (c >> 5), columns m0 + 4 (c & 31) .. +3,
  // so 32 lanes read one contiguous 512-byte row segment.
  constexpr int WCH = (MODE == GEMM_WGRAD) ? BM * BN / 4 / NTHR : 1;
  f32x4 wpre[WCH];
  // Workgroup-uniform tile bases; lanes add a 32-bit offset (row * M + col).
  float* wtile = master + g.w_off + static_cast<int64_t>(n0) * M + m0;
  const float* wtile_in = master_in + g.w_off + static_cast<int64_t>(n0) * M + m0;
  if constexpr (MODE == GEMM_WGRAD) {
#pragma unroll
    for (int p = 0; p < WCH; ++p) {
      const int c = tid + NTHR * p, row = c >> 5, col = 4 * (c & 31);
      const bool ok = n0 + row < N && m0 + col < M;  // M % 4 == 0: chunks are whole
      wpre[p] = ok ? __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(wtile_in + (row * M + col)))
                   : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }
  }

  f32x16 acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
  // Non-split forward / backward-data: sum of the finished chunks.
  constexpr bool TOTAL = CHUNKED && !SPLIT;
  f32x16 tot[TOTAL ? MI : 1][TOTAL ? NJ : 1];

  // Backward-weight bias: db[o] = sum_b delta[b][o] in blocks of 64 batch
  // rows, each block row by row (dcur), block sums left to right (dbias).
  const bool bias_wg = (MODE == GEMM_WGRAD) && m0 == 0;
  float dbias = 0.0f, dcur = 0.0f;

  // A: rows m (RowTile, FWD) or k rows with m chunks (TransTile).
  // B: rows n (RowTile, FWD / DGRAD) or k rows with n chunks (TransTile, WGRAD).
#define LOAD_A(t, k0)                                                     \
  do {                                                                    \
    if constexpr (MODE == GEMM_FWD) t.load(sa, A, k0, g.a_ext, tid);      \
    else t.load(A, g.a_ld, m0, g.a_ext, k0, K, tid);                      \
  } while (0)
#define LOAD_B(t, k0)                                                     \
  do {                                                                    \
    if constexpr (MODE == GEMM_WGRAD) t.load(B, g.b_ld, n0, g.b_ext, k0, K, tid); \
    else {                                                                \
      t.load(sb, B, k0, g.b_ext, tid);                                    \
      if (GATHER && (k0) < kend && ((k0) / BK) % gm == mt)                \
        t.copy_out(rows_out, g.rows_out_ld, n0, N, k0, g.b_ext, tid);     \
    }                                                                     \
  } while (0)

  auto compute = [&](int buf) {
    mma_tile<BF16, MI, NJ>(lds_a(buf), lds_b(buf), wm, wn, lane, acc);
    if (bias_wg && tid < BN) {
      // db[o] = sum_b delta[b][o]: row tid of the B tile, in k order.
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(lds_b(buf) + lds_word(tid, c));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if constexpr (BF16) {
            dcur += __uint_as_float(v[e] << 16);
            dcur += __uint_as_float(v[e] & 0xFFFF0000u);
          } else {
            dcur += __uint_as_float(v[e]);
          }
        }
      }
    }
  };

  // After K tile j (counted from kbeg): close the 64-row bias block it ends.
  auto fold = [&](int j, int nk) {
    if constexpr (MODE == GEMM_WGRAD) {
      static_assert(64 % BK == 0, "64-row bias blocks of whole K tiles");
      if (((j + 1) * BK) % 64 == 0 || j + 1 == nk) {
        dbias = j * BK < 64 ? dcur : dbias + dcur;
        dcur = 0.0f;
      }
    }
  };
  // After the last K tile of a chunk: its sum into tot.  Called once per
  // chunk from outside the tile loop (tested inside it, the fold became
  // selects that ran at every tile).
  auto fold_chunk = [&](bool first) {
    if constexpr (TOTAL) {
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) {
          tot[i][jj] = first ? acc[i][jj] : tot[i][jj] + acc[i][jj];
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[i][jj][r] = 0.0f;
        }
    }
  };
  // tiles [j0, chunk_end(j0)): one chunk with chunk totals, else all of K
  auto chunk_end = [&](int j0, int nk) { return TOTAL ? (nk - j0 < TPC ? nk : j0 + TPC) : nk; };

  // Loads past the end of K read zeros, so the loop bodies are straight-line.
  const int nk = (kend - kbeg + BK - 1) / BK;
  if constexpr (S::ST == 1) {
    // One register stage, LDS double buffer (always for the short K of the
    // backward-weight pass, the batch).
    LOAD_A(ta, kbeg);
    LOAD_B(tb, kbeg);
    ta.store(lds_a(0), tid);
    tb.store(lds_b(0), tid);
    __syncthreads();
    for (int j0 = 0; j0 < nk;) {
      const int jend = chunk_end(j0, nk);
      for (int kt = j0; kt < jend; ++kt) {
        const int buf = kt & 1;
        LOAD_A(ta, kbeg + (kt + 1) * BK);
        LOAD_B(tb, kbeg + (kt + 1) * BK);
        compute(buf);
        fold(kt, nk);
        ta.store(lds_a(buf ^ 1), tid);
        tb.store(lds_b(buf ^ 1), tid);
        __syncthreads();
      }
      fold_chunk(jend <= TPC);
      j0 = jend;
    }
  } else {
    // ST register stages: while tile j is multiplied out of LDS buffer j & 1,
    // tiles j+1 .. j+ST are loading into the register sets t*[(j+1) % ST] ..
    // The loop is unrolled by ST so every register set is indexed statically.
    constexpr int ST = S::ST;
    decltype(ta) tA[ST];
    decltype(tb) tB[ST];
#pragma unroll
    for (int u = 0; u < ST; ++u) {
      LOAD_A(tA[u], kbeg + u * BK);
      LOAD_B(tB[u], kbeg + u * BK);
    }
    tA[0].store(lds_a(0), tid);
    tB[0].store(lds_b(0), tid);
    __syncthreads();
    static_assert(!TOTAL || TPC % ST == 0, "chunks start on register set 0");
    auto tile_step = [&](int j, auto uc) {
      constexpr int u = decltype(uc)::value;
      LOAD_A(tA[u], kbeg + (j + ST) * BK);
      LOAD_B(tB[u], kbeg + (j + ST) * BK);
      compute(j & 1);
      fold(j, nk);
      tA[(u + 1) % ST].store(lds_a((j + 1) & 1), tid);
      tB[(u + 1) % ST].store(lds_b((j + 1) & 1), tid);
      __syncthreads();
    };
    // Whole groups of ST tiles in the loops (no exit between the tiles of a
    // group, so every path into the loop header has the same loads in
    // flight: with an exit after any tile the compiler waited for every load
    // at the header, halving the prefetch distance); a last tile of K that
    // does not fill a group comes after.
    static_assert(ST == 2, "two register sets");
    const int nkg = nk - nk % ST;
    for (int j0 = 0; j0 < nkg;) {
      const int jc = chunk_end(j0, nk), jend = jc < nkg ? jc : nkg;
      for (int kt = j0; kt < jend; kt += ST) {
        tile_step(kt, Ic<0>());
        tile_step(kt + 1, Ic<1>());
      }
      if (jend == jc) fold_chunk(jend <= TPC);
      j0 = jend;
    }
    if (nkg < nk) {
      tile_step(nkg, Ic<0>());
      fold_chunk(nk <= TPC);
    }
  }
#undef LOAD_A
#undef LOAD_B

  if constexpr (MODE == GEMM_WGRAD) {
    static_assert(BM == 128 && BN == 128, "update epilogue layout");
    // dW tile -> LDS as [o][i] (row n - n0, 16-byte chunk (m - m0) / 4 placed
    // at chunk ^ (row & 31)), then every thread updates the chunks it
    // prefetched: coalesced master read/write and bf16 refresh.
    float* dws = reinterpret_cast<float*>(lds_all);  // all 64 KB of LDS
    auto dw_at = [](int row, int ch) { return row * BM + ((ch ^ (row & 31)) << 2); };
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = ncol(j) - n0, ch = (mrow(i, q) - m0) >> 2;
          *reinterpret_cast<f32x4*>(dws + dw_at(row, ch)) =
              f32x4{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                    acc[i][j][4 * q + 3]};
        }
    __syncthreads();
    uint16_t* ctile = (g.wcopy && z < g.wcopy_slots)
                          ? g.wcopy + z * g.wcopy_slot + g.w_off + static_cast<int64_t>(n0) * M + m0
                          : nullptr;
#pragma unroll
    for (int p = 0; p < WCH; ++p) {
      const int c = tid + NTHR * p, row = c >> 5, col = 4 * (c & 31);
      if (n0 + row < N && m0 + col < M) {
        const f32x4 d = *reinterpret_cast<const f32x4*>(dws + dw_at(row, c & 31));
        f32x4 w = wpre[p];
        for (int e = 0; e < 4; ++e) w[e] = fmaf(-g.lr, d[e], w[e]);
        const int at = row * M + col;
        __builtin_nontemporal_store(w, reinterpret_cast<f32x4*>(wtile + at));
        if (ctile) {
          u32x2 o;
          o[0] = f2bf(w[0]) | (f2bf(w[1]) << 16);
          o[1] = f2bf(w[2]) | (f2bf(w[3]) << 16);
          __builtin_nontemporal_store(o, reinterpret_cast<u32x2*>(ctile + at));
        }
      }
    }
    if (bias_wg && tid < BN && n0 + tid < N)
      master[g.b_off + n0 + tid] = fmaf(-g.lr, dbias, master_in[g.b_off + n0 + tid]);
    return;
  } else if constexpr (SPLIT) {
    // Partial `chunk` of outputs (m, n): fp32 at part[slot][chunk][n][m]
    // (row stride out_ld; columns up to round_up(M, 4) stay inside it).
    float* part = g.part + z * g.part_slot + static_cast<int64_t>(chunk) * N * g.out_ld;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int n = ncol(j);
        if (n >= N) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int m = mrow(i, q);
          if (m >= M) continue;
          *reinterpret_cast<f32x4*>(part + static_cast<int64_t>(n) * g.out_ld + m) =
              f32x4{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                    acc[i][j][4 * q + 3]};
        }
      }
    return;
  } else {
    // Epilogue over groups of four consecutive rows m..m+3 at column n: the
    // inputs (bias / mask) of every group first, loads in flight together
    // (outside the outputs row 0, column 0 is read and not used), then the
    // stores.
    f32x4 ea[MI][NJ][4];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int n = ncol(j);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int m = mrow(i, q);
          const bool in = n < N && m < M;
          ea[i][j][q] = epi_load<BF16, MODE>(g, z, in ? n : 0, in ? m : 0,
                                             in ? ((M - m >= 4) ? 4 : M - m) : 4, master_in);
        }
      }
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int n = ncol(j);
        if (n >= N) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int m = mrow(i, q);
          if (m >= M) continue;
          const int cnt = (M - m >= 4) ? 4 : M - m;
          store_out_with<BF16, MODE>(g, z, n, m, cnt,
                                     f32x4{tot[i][j][4 * q], tot[i][j][4 * q + 1],
                                           tot[i][j][4 * q + 2], tot[i][j][4 * q + 3]},
                                     ea[i][j][q]);
        }
      }
  }
}

// ---------------------------------------------------------------------------
// Forward / backward-data of bf16 models with whole-batch tiles (W, V): K
// tiles go from global memory straight into LDS (global_load_lds, 16 bytes
// per lane), ST stages deep, so no VGPRs hold tiles in flight and ST - 1
// stages load while one is multiplied.  One wave instruction fills 8 LDS rows
// (1 KB, lane l at byte 16 l); the swizzle is applied on the source side:
// the lane at physical chunk p of tile row r reads logical chunk
// p ^ ((r ^ r >> 3) & 7).  Backward-data's weight operand is stored
// M-contiguous and is transposed through registers as in gemm_kernel, one
// stage ahead.  The summation order is that of gemm_kernel.

typedef __attribute__((address_space(1))) void global_void;
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ void dma16(const void* src, uint32_t* lds_row) {
  __builtin_amdgcn_global_load_lds((global_void*)src, (lds_void*)lds_row, 16, 0, 0);
}

// Wait until at most N vector memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// LDS writes of this wave done, then the workgroup barrier.  The barrier is
// opaque to the compiler (no memory operation moves across it) and, unlike
// __syncthreads, does not wait for the loads still streaming into LDS.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4));  // lgkmcnt(0)
  asm volatile("s_barrier" ::: "memory");
}

template <int NTHR, int ROWS>
struct DmaTile {
  static constexpr int P = ROWS * 8 / NTHR;
  static_assert(ROWS * 8 % NTHR == 0 && NTHR % 64 == 0, "whole wave instructions");
  const uint16_t* src[P];
  const void* zero;  // the zero source, its address taken once
  bool ok[P];
  int kc[P];
  __device__ __forceinline__ void init(const uint16_t* base, int64_t ld, const int32_t* gather,
                                       int row0, int R, int tid) {
    zero = k_zero16;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int idx = tid + NTHR * p, r = idx >> 3;
      const int lc = (idx & 7) ^ ((r ^ (r >> 3)) & 7);
      const int gr = row0 + r;
      ok[p] = gr < R;
      const int grc = gr < R ? gr : R - 1;
      const int64_t row = gather ? gather[grc] : grc;
      kc[p] = 8 * lc;
      src[p] = base + row * ld + 8 * lc;
    }
  }
  // P wave instructions; wave w's instruction p fills tile rows
  // (64 w + NTHR p) / 8 .. + 7.
  __device__ __forceinline__ void issue_one(int p, uint32_t* tile, int k0, int ext, int tid) const {
    const bool in = ok[p] && k0 + kc[p] < ext;
    dma16(in ? static_cast<const void*>(src[p] + k0) : zero,
          tile + (((tid & ~63) + NTHR * p) >> 3) * ROW_U32);
  }
  __device__ __forceinline__ void issue(uint32_t* tile, int k0, int ext, int tid) const {
#pragma unroll
    for (int p = 0; p < P; ++p) issue_one(p, tile, k0, ext, tid);
  }
};

template <int MODE, bool GATHER, int SID, bool SPLIT>
__global__ __launch_bounds__((ShapeOf<MODE, SID>::type::NT), (ShapeOf<MODE, SID>::type::MIN_WAVES)) void
gemm_dma_kernel(GemmArgs g) {
  typedef uint16_t T;
  typedef typename ShapeOf<MODE, SID>::type S;
  static_assert(MODE == GEMM_FWD || MODE == GEMM_DGRAD, "forward / backward-data only");
  constexpr int NTHR = S::NT, WAVES_N = S::WAVES_N, MI = S::MI, NJ = S::NJ;
  constexpr int BM = S::BM, BN = S::BN, NS = S::ST;
  constexpr int BK = El<true>::BK;
  constexpr int TPC = KCHUNK / BK;
  static_assert(NS >= 2, "at least one stage loading while one is used");
  __shared__ __attribute__((aligned(16))) uint32_t lds_all[NS * (BM + BN) * ROW_U32];
  auto lds_a = [&](int buf) { return lds_all + buf * BM * ROW_U32; };
  auto lds_b = [&](int buf) { return lds_all + NS * BM * ROW_U32 + buf * BN * ROW_U32; };

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N, h = lane >> 5;
  const int work = xcd_work(blockIdx.y * gridDim.x + blockIdx.x, gridDim.x * gridDim.y);
  const int z = work / gridDim.x;
  const int rep = g.order[z];
  const int M = g.M, N = g.N, K = g.K;
  const int gn = (N + BN - 1) / BN;
  const int t = work % gridDim.x;
  const int nchunks = (K + KCHUNK - 1) / KCHUNK;
  const int tiles = SPLIT ? static_cast<int>(gridDim.x) / nchunks : static_cast<int>(gridDim.x);
  const int chunk = SPLIT ? t / tiles : 0, tile = SPLIT ? t % tiles : t;
  const int m0 = (tile / gn) * BM, n0 = (tile % gn) * BN;
  const int kbeg = SPLIT ? chunk * KCHUNK : 0;
  const int kend = SPLIT ? (K - kbeg < KCHUNK ? K : kbeg + KCHUNK) : K;
  const int nk = (kend - kbeg + BK - 1) / BK;

  const T* A = static_cast<const T*>(g.a) + (g.a_by_order ? rep : z) * g.a_slot;
  const T* B = static_cast<const T*>(g.b) + z * g.b_slot;
  const float* master_in = g.master_in + static_cast<int64_t>(rep) * g.master_in_slot;
  T* rows_out = GATHER ? static_cast<T*>(g.rows_out) + z * g.rows_out_slot : nullptr;
  const int gm = (M + BM - 1) / BM, mt = m0 / BM;

  DmaTile<NTHR, BN> db;
  db.init(B, g.b_ld, GATHER ? g.gather + z * g.gather_slot : nullptr, n0, N, tid);
  DmaTile<NTHR, BM> da;             // FWD: weights, K-contiguous
  TransTile<true, NTHR, BM> ta[2];  // DGRAD: weights, M-contiguous, via registers, two ahead
  if constexpr (MODE == GEMM_FWD) da.init(A, g.a_ld, nullptr, m0, M, tid);

  f32x16 acc[MI][NJ], tot[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  auto k_of = [&](int s) { return kbeg + s * BK; };
  // FWD issues stage s as A then B (PA + PB instructions per thread);
  // DGRAD loads A(s) into registers and issues B(s) (2 + PB).
  constexpr int PA = MODE == GEMM_FWD ? DmaTile<NTHR, BM>::P : 2 * TransTile<true, NTHR, BM>::P;
  constexpr int PB = DmaTile<NTHR, BN>::P;
  auto issue_b = [&](int s) { db.issue(lds_b(s % NS), k_of(s), g.b_ext, tid); };

  if constexpr (MODE == GEMM_FWD) {
#pragma unroll
    for (int s = 0; s < NS - 1; ++s) {
      da.issue(lds_a(s), k_of(s), g.a_ext, tid);
      issue_b(s);
    }
  } else {
    // A(0) .. A(NS - 2) into LDS, B(0) .. B(NS - 2) streaming, A(NS - 1) and
    // A(NS) loading into the two register tiles; A(NS) and B(NS - 2) are the
    // operations of "step -1".
    static_assert(NS >= 3, "B(j) is older than the last step's operations");
#pragma unroll
    for (int s = 0; s < NS - 1; ++s) {
      ta[0].load(A, g.a_ld, m0, g.a_ext, k_of(s), K, tid);
      wait_vm<0>();
      ta[0].store(lds_a(s), tid);
    }
#pragma unroll
    for (int s = 0; s < NS - 2; ++s) issue_b(s);
    ta[(NS - 1) & 1].load(A, g.a_ld, m0, g.a_ext, k_of(NS - 1), K, tid);
    ta[NS & 1].load(A, g.a_ld, m0, g.a_ext, k_of(NS), K, tid);
    issue_b(NS - 2);
  }

  // Step j.  The register tile of A(j + NS - 1) is ta[(j + NS - 1) & 1]:
  // the loop runs pairs of steps so that the index is static.
  auto step = [&](int j, auto par) {
    // Stage j landed.  FWD: stages j + 1 .. j + NS - 2 stay in flight.
    // DGRAD: A(j + NS - 1) in registers too (issued two steps ago); the
    // last step's A(j + NS) and B(j + NS - 2) stay in flight.
    if constexpr (MODE == GEMM_FWD) wait_vm<(NS - 2) * (PA + PB)>();
    else wait_vm<PA + PB>();
    lds_barrier();
    // DGRAD: nothing that reads the register tile moves above the wait (the
    // compiler would then wait for every load at the top of the loop)
    if constexpr (MODE == GEMM_DGRAD) ta[decltype(par)::value].pin();
    const int k0 = k_of(j);
    if (GATHER && k0 < kend && (k0 / BK) % gm == mt) {
      // Layer 1: this workgroup keeps K tile j of the gathered batch rows.
      constexpr int PC = BN * 8 / NTHR;
#pragma unroll
      for (int p = 0; p < PC; ++p) {
        const int idx = tid + NTHR * p, row = idx >> 3, c = idx & 7, k = k0 + 8 * c;
        const u32x4 v = *reinterpret_cast<const u32x4*>(lds_b(j % NS) + lds_word(row, c));
        if (n0 + row < N && k < g.b_ext)
          *reinterpret_cast<u32x4*>(rows_out + static_cast<int64_t>(n0 + row) * g.rows_out_ld + k) = v;
      }
      wait_vm<0>();
    }
    if constexpr (MODE == GEMM_DGRAD) {
      // A(j + NS - 1) from registers into its LDS buffer (last read by the
      // product of tile j - 1, before the barrier), then load A(j + NS + 1)
      // into the same registers.
      constexpr int R = decltype(par)::value;
      ta[R].store(lds_a((j + NS - 1) % NS), tid);
      ta[R].load(A, g.a_ld, m0, g.a_ext, k_of(j + NS + 1), K, tid);
      issue_b(j + NS - 1);
      mma_tile<true, MI, NJ>(lds_a(j % NS), lds_b(j % NS), wm, wn, lane, acc);
    } else if constexpr (SPLIT) {
      // split-K tiles (few workgroups, latency-bound): the whole stage first
      da.issue(lds_a((j + NS - 1) % NS), k_of(j + NS - 1), g.a_ext, tid);
      issue_b(j + NS - 1);
      mma_tile<true, MI, NJ>(lds_a(j % NS), lds_b(j % NS), wm, wn, lane, acc);
    } else {
      // stage j + NS - 1: its PA + PB instructions spread over the four k
      // groups of this step, each issued behind the group's operand reads so
      // that the products start without waiting for the whole stage's issue
      uint32_t* const na = lds_a((j + NS - 1) % NS);
      uint32_t* const nb = lds_b((j + NS - 1) % NS);
      const int kn = k_of(j + NS - 1);
      mma_tile<true, MI, NJ>(lds_a(j % NS), lds_b(j % NS), wm, wn, lane, acc, [&](int s) {
#pragma unroll
        for (int q = 0; q < PA + PB; ++q) {
          if (q * 4 / (PA + PB) != s) continue;
          if (q < PA) da.issue_one(q, na, kn, g.a_ext, tid);
          else db.issue_one(q - PA, nb, kn, g.b_ext, tid);
        }
      });
    }
  };
  // The steps chunk by chunk (TPC steps each, even: the register-tile index of
  // a chunk's first step is always that of step 0), the chunk's sum folded into
  // tot after its last step.  (A fold tested inside every step was turned into
  // selects the compiler ran at every step: some 400 VALU instructions per 32
  // MFMAs.)
  static_assert(TPC % 2 == 0, "chunks of an even number of K tiles");
  int j = 0;
  while (j < nk) {
    const int jend = nk - j < TPC ? nk : j + TPC;
    for (; j + 1 < jend; j += 2) {
      step(j, Ic<(NS - 1) & 1>());
      step(j + 1, Ic<NS & 1>());
    }
    if (j < jend) {
      step(j, Ic<(NS - 1) & 1>());
      ++j;
    }
    if constexpr (!SPLIT) {
      const bool first = jend <= TPC;
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) {
          tot[i][jj] = first ? acc[i][jj] : tot[i][jj] + acc[i][jj];
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[i][jj][e] = 0.0f;
        }
    }
  }
  wait_vm<0>();  // nothing streams into LDS past the end of the workgroup

  auto mrow = [&](int i, int q) { return m0 + wm * 32 * MI + 32 * i + 8 * q + 4 * h; };
  auto ncol = [&](int j) { return n0 + wn * 32 * NJ + 32 * j + (lane & 31); };
  if constexpr (SPLIT) {
    float* part = g.part + z * g.part_slot + static_cast<int64_t>(chunk) * N * g.out_ld;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int n = ncol(j);
        if (n >= N) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int m = mrow(i, q);
          if (m >= M) continue;
          *reinterpret_cast<f32x4*>(part + static_cast<int64_t>(n) * g.out_ld + m) =
              f32x4{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                    acc[i][j][4 * q + 3]};
        }
      }
  } else {
    // the epilogue's inputs (bias / mask) of every group first, so that their
    // loads are in flight together, then the stores
    f32x4 ea[MI][NJ][4];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int n = ncol(j);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          // outside the outputs: row 0, column 0 is read instead (no branch
          // around the load) and not used
          const int m = mrow(i, q);
          const bool in = n < N && m < M;
          ea[i][j][q] = epi_load<true, MODE>(g, z, in ? n : 0, in ? m : 0,
                                             in ? ((M - m >= 4) ? 4 : M - m) : 4, master_in);
        }
      }
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int n = ncol(j);
        if (n >= N) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int m = mrow(i, q);
          if (m >= M) continue;
          const int cnt = (M - m >= 4) ? 4 : M - m;
          store_out_with<true, MODE>(g, z, n, m, cnt,
                                     f32x4{tot[i][j][4 * q], tot[i][j][4 * q + 1],
                                           tot[i][j][4 * q + 2], tot[i][j][4 * q + 3]},
                                     ea[i][j][q]);
        }
      }
  }
}

// ---------------------------------------------------------------------------
// Backward-weight + SGD update of bf16 models.  Both operands are stored
// with the batch (K) slowest, act[b][i] and delta[b][o]; their K tiles go
// into LDS unchanged (global_load_lds, 16 bytes per lane, 4 rows of 256
// bytes per wave instruction) and are transposed on the way out by
// ds_read_b64_tr_b16.  Within each 16-lane group that read returns to lane
// 4a + b element e the element b of the 4 that lane a + 4e addressed; when
// lane a + 4e addresses row k0 + e, columns c0 + 4a .. + 3, lane j receives
// rows k0 .. k0 + 3 of column c0 + j, i.e. four consecutive K of one MFMA
// row.  Two such reads give the 8 K of a 32x32x16 operand lane, in the
// order of gemm_kernel, so the sums are the same.  Tile rows are 256 bytes;
// the 16-byte chunk c of row k sits at c ^ 4 (k & 3), which spreads the
// transposing reads of 4 consecutive rows over all chunk positions.
// Tile 128 (in) x 128 (out), 4 waves of 64 x 64, K tiles of 32 rows,
// 3 stages (48 KB of LDS); the update epilogue stages dW through LDS in two
// halves of 64 output rows (32 KB), so that three workgroups fit a CU.
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

__device__ __forceinline__ int trow_chunk(int k, int c) { return c ^ ((k & 3) << 2); }

template <int ROWS_PER_STAGE, int COLS>
struct DmaRowsTile {  // K rows x COLS bf16 (COLS * 2 = 256 bytes per row)
  static_assert(COLS == 128, "256-byte rows");
  static constexpr int P = ROWS_PER_STAGE / 16;  // wave instructions per thread, 4 waves
  const uint16_t* src[P];
  int row[P];
  bool colok[P];
  __device__ __forceinline__ void init(const uint16_t* base, int64_t ld, int col0, int ext,
                                       int tid) {
    const int w = tid >> 6, l = tid & 63;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const int r = 4 * (w + 4 * p) + (l >> 4);
      const int c = trow_chunk(r, l & 15);
      row[p] = r;
      colok[p] = col0 + 8 * c < ext;
      src[p] = base + r * ld + col0 + 8 * c;
    }
  }
  __device__ __forceinline__ void issue(uint32_t* tile, int k0, int K, int64_t ld, int tid) const {
    const int w = tid >> 6;
#pragma unroll
    for (int p = 0; p < P; ++p) {
      const bool in = colok[p] && k0 + row[p] < K;
      dma16(in ? static_cast<const void*>(src[p] + static_cast<int64_t>(k0) * ld)
               : static_cast<const void*>(k_zero16),
            tile + 4 * (w + 4 * p) * 64);
    }
  }
};

// MFMA operand (8 consecutive K of column col0 + (lane & 31)) from a tile of
// 256-byte rows, K rows k0 + 8 h .. + 7.  The two transposing reads are
// inline asm: after an LDS-DMA load the compiler waits for every vector memory
// operation in flight (vmcnt(0)) before a ds_read_b64_tr_b16 it emits itself,
// which drained the next stages' loads at every K step.  The compiler does
// not wait for these reads either: the caller waits (lgkmcnt) before using
// the operands, through an asm statement that takes them as operands.
__device__ __forceinline__ bf16x8 tr_operand(const uint32_t* tile, int k0, int col0, int lane) {
  const int g = lane >> 4, il = lane & 15, a = il & 3, e = il >> 2, h = lane >> 5;
  const int col = col0 + 16 * (g & 1) + 4 * a;
  u32x2 v[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int k = k0 + 8 * h + 4 * q + e;
    const int byte = k * 256 + trow_chunk(k, col >> 3) * 16 + (col & 4) * 2;
    const uint32_t addr = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(
        (const __attribute__((address_space(3))) char*)(reinterpret_cast<const char*>(tile) + byte)));
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v[q]) : "v"(addr));
  }
  const u32x4 all = {v[0][0], v[0][1], v[1][0], v[1][1]};
  return __builtin_bit_cast(bf16x8, all);
}

// PRE: master chunks per thread fetched before the products (the tile has
// 16); the others are fetched when the epilogue starts, which keeps
// registers for a third workgroup per CU.
template <int MINW, int PRE>
__global__ __launch_bounds__(256, MINW) void wgrad_dma_kernel(GemmArgs g) {
  constexpr int BM = 128, BN = 128, BK = 32, NS = 3, NTHR = 256, MI = 2, NJ = 2;
  constexpr int STAGE_U32 = BK * 256 / 4;  // one operand stage: 32 rows x 256 bytes
  __shared__ __attribute__((aligned(16))) uint32_t lds_all[2 * NS * STAGE_U32];
  auto lds_a = [&](int buf) { return lds_all + buf * STAGE_U32; };
  auto lds_b = [&](int buf) { return lds_all + (NS + buf) * STAGE_U32; };

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, h = lane >> 5;
  const int work = xcd_work(blockIdx.y * gridDim.x + blockIdx.x, gridDim.x * gridDim.y);
  const int z = work / gridDim.x;
  const int rep = g.order[z];
  const int M = g.M, N = g.N, K = g.K;
  const int gn = (N + BN - 1) / BN;
  const int t = work % gridDim.x;
  const int m0 = (t / gn) * BM, n0 = (t % gn) * BN;

  const uint16_t* A = static_cast<const uint16_t*>(g.a) + z * g.a_slot;
  const uint16_t* B = static_cast<const uint16_t*>(g.b) + z * g.b_slot;
  float* master = g.master + static_cast<int64_t>(rep) * g.master_slot;
  const float* master_in = g.master_in + static_cast<int64_t>(rep) * g.master_in_slot;

  DmaRowsTile<BK, BM> da;
  DmaRowsTile<BK, BN> db;
  da.init(A, g.a_ld, m0, g.a_ext, tid);
  db.init(B, g.b_ld, n0, g.b_ext, tid);
  constexpr int PS = DmaRowsTile<BK, BM>::P + DmaRowsTile<BK, BN>::P;  // per stage and thread
  auto issue = [&](int s) {
    da.issue(lds_a(s % NS), s * BK, K, g.a_ld, tid);
    db.issue(lds_b(s % NS), s * BK, K, g.b_ld, tid);
  };
  issue(0);
  issue(1);

  // fp32 master tile W[n0 .. n0 + 127][m0 .. m0 + 127], issued after the
  // first two operand stages: chunk c = tid + 256 p is row n0 + (c >> 5),
  // columns m0 + 4 (c & 31) .. + 3 (32 lanes read one 512-byte row segment).
  constexpr int WCH = BM * BN / 4 / NTHR;  // chunks per thread, both halves
  static_assert(PRE >= 0 && PRE <= WCH, "prefetch depth");
  f32x4 wpre[PRE > 0 ? PRE : 1];
  float* wtile = master + g.w_off + static_cast<int64_t>(n0) * M + m0;
  const float* wtile_in = master_in + g.w_off + static_cast<int64_t>(n0) * M + m0;
  auto master_chunk = [&](int p) {
    const int c = tid + NTHR * p, row = c >> 5, col = 4 * (c & 31);
    const bool ok = n0 + row < N && m0 + col < M;  // M % 4 == 0: chunks are whole
    return __builtin_nontemporal_load(
        reinterpret_cast<const f32x4*>(ok ? wtile_in + (row * M + col)
                                          : reinterpret_cast<const float*>(k_zero16)));
  };
#pragma unroll
  for (int p = 0; p < PRE; ++p) wpre[p] = master_chunk(p);

  f32x16 acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
  // bias: 64-row blocks (two stages) row by row, block sums left to right
  const bool bias_wg = m0 == 0;
  float dbias = 0.0f, dcur = 0.0f;

  const int nk = (K + BK - 1) / BK;
  for (int j = 0; j < nk; ++j) {
    // Stage j landed; in flight after it: stage j + 1 and, until stage 2 is
    // waited for, the master tile (issued between stages 1 and 2).
    if (j < 2) wait_vm<PS + PRE>();
    else wait_vm<PS>();
    lds_barrier();
    issue(j + 2);
    const uint32_t* As = lds_a(j % NS);
    const uint32_t* Bs = lds_b(j % NS);
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      bf16x8 a[MI], b[NJ];
#pragma unroll
      for (int i = 0; i < MI; ++i) a[i] = tr_operand(As, 16 * s, wm * 64 + 32 * i, lane);
#pragma unroll
      for (int jj = 0; jj < NJ; ++jj) b[jj] = tr_operand(Bs, 16 * s, wn * 64 + 32 * jj, lane);
      // the operand reads done (tr_operand); the products depend on this wait
      static_assert(MI == 2 && NJ == 2, "the wait names the four operands");
      asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a[0]), "+v"(a[1]), "+v"(b[0]), "+v"(b[1]));
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj)
          acc[i][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[jj], acc[i][jj], 0, 0, 0);
    }
    if (bias_wg && tid < BN) {
      // db[o] = sum_b delta[b][o], column tid of this stage, in K order.
      const char* bs = reinterpret_cast<const char*>(Bs);
#pragma unroll 8
      for (int r = 0; r < BK; ++r) {
        const uint16_t v = *reinterpret_cast<const uint16_t*>(
            bs + r * 256 + trow_chunk(r, tid >> 3) * 16 + (tid & 7) * 2);
        dcur += __uint_as_float(static_cast<uint32_t>(v) << 16);
      }
      static_assert(64 % BK == 0, "64-row bias blocks of whole stages");
      if (((j + 1) * BK) % 64 == 0 || j + 1 == nk) {
        dbias = j * BK < 64 ? dcur : dbias + dcur;
        dcur = 0.0f;
      }
    }
  }
  wait_vm<0>();  // trailing stages and the master tile
  lds_barrier();  // every wave done with the operand stages

  // Epilogue in two halves of 64 output rows: the waves holding those rows
  // store dW^T to LDS as [o][i] (row n - n0 - 64 half, 16-byte chunk
  // (m - m0) / 4 placed at chunk ^ (row & 31)), then every thread updates
  // the master chunks of that half it prefetched.
  float* dws = reinterpret_cast<float*>(lds_all);  // 64 rows x 512 bytes
  auto dw_at = [](int row, int ch) { return row * BM + ((ch ^ (row & 31)) << 2); };
  uint16_t* ctile = (g.wcopy && z < g.wcopy_slots)
                        ? g.wcopy + z * g.wcopy_slot + g.w_off + static_cast<int64_t>(n0) * M + m0
                        : nullptr;
  f32x4 wlate[WCH - PRE > 0 ? WCH - PRE : 1];
  if constexpr (PRE < WCH) {
#pragma unroll
    for (int p = PRE; p < WCH; ++p) wlate[p - PRE] = master_chunk(p);
  }
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    if (wn == half) {
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int row = 32 * jj + (lane & 31);  // n - n0 - 64 half
            const int ch = (wm * 64 + 32 * i + 8 * q + 4 * h) >> 2;
            *reinterpret_cast<f32x4*>(dws + dw_at(row, ch)) =
                f32x4{acc[i][jj][4 * q], acc[i][jj][4 * q + 1], acc[i][jj][4 * q + 2],
                      acc[i][jj][4 * q + 3]};
          }
    }
    __syncthreads();
#pragma unroll
    for (int p = half * WCH / 2; p < (half + 1) * WCH / 2; ++p) {
      const int c = tid + NTHR * p, row = c >> 5, col = 4 * (c & 31);
      if (n0 + row < N && m0 + col < M) {
        const f32x4 d = *reinterpret_cast<const f32x4*>(dws + dw_at(row - 64 * half, c & 31));
        f32x4 w = p < PRE ? wpre[p < PRE ? p : 0] : wlate[p >= PRE ? p - PRE : 0];
        (void)wpre;
        for (int e = 0; e < 4; ++e) w[e] = fmaf(-g.lr, d[e], w[e]);
        const int at = row * M + col;
        __builtin_nontemporal_store(w, reinterpret_cast<f32x4*>(wtile + at));
        if (ctile) {
          u32x2 o;
          o[0] = f2bf(w[0]) | (f2bf(w[1]) << 16);
          o[1] = f2bf(w[2]) | (f2bf(w[3]) << 16);
          __builtin_nontemporal_store(o, reinterpret_cast<u32x2*>(ctile + at));
        }
      }
    }
    if (half == 0) __syncthreads();
  }
  if (bias_wg && tid < BN && n0 + tid < N)
    master[g.b_off + n0 + tid] = fmaf(-g.lr, dbias, master_in[g.b_off + n0 + tid]);
}

// ---------------------------------------------------------------------------
// Backward pass of a hidden layer (l >= 2) of a bf16 model in one kernel:
// backward-data, backward-weight and the SGD update of Eq. 4.  A workgroup
// owns a strip of 64 input features i (columns of W_l) and walks the output
// features o in chunks of 64.  For each chunk it streams the fp32 master rows
// of its strip, rounds them to the bf16 working weights Wq = bf16(W) the
// forward pass used, and computes
//   backward-data    C[i][b] += sum_{o in chunk} Wq[o][i] delta[b][o]
//   backward-weight  dW[o][i] = sum_b act[b][i] delta[b][o]
//   update           W <- W - eta dW (fp32 master, bf16 copy refreshed);
//                    the strip t % strips also updates the chunk's bias,
//                    b <- b - eta sum_b delta.
// Backward-data thus reads no weights of its own: its products ride on the
// master stream of the update.  Its result is masked by act > 0 and stored
// as the bf16 delta of the layer below.
//
// Two roles of four waves each, one barrier per chunk step:
//   stream waves (0-3) at step t stage chunk t + 1 into LDS (delta, and Wq
//     rounded from the master rows), issue the loads of chunk t + 3 (delta)
//     and t + 4 (master), and apply dW of chunk t - 1 to its master rows;
//   math waves (4-7) at step t run the MFMA products of chunk t and leave dW
//     in LDS.
// Every SIMD holds one wave of each role, so the update's vector work and
// memory traffic overlap the products.  The stream waves' loads and stores
// go through buffer resources (out-of-range offsets read zeros and write
// nothing), so their loop has no branches around memory operations.
//
// The summation orders are those of the separate kernels: backward-data sums
// o in chunks of KCHUNK (each from zero, 16 at a time, chunk sums left to
// right); backward-weight sums the batch 16 rows at a time from zero; the
// bias sums blocks of 64 batch rows row by row and the block sums left to
// right.  The operand roles of every MFMA are those of the separate kernels
// too.  Backward-weight runs over 128 or 256 batch rows (zero past B) where
// the separate kernel stops at the batch rounded up to 32; the extra zero
// products can only turn a dW of -0 into +0, which changes the updated
// weight only when that weight is -0 itself.
// SPLIT: a workgroup covers `cps` KCHUNK ranges of o and stores the
// backward-data sum of each as that chunk's partial; splitk_reduce_kernel
// finishes.
// DG = false: backward-weight and the update only (layer 1, whose input needs
// no gradient): no Wq stage, no backward-data products; a split then needs
// no partials.  The update streams the master the same way, which on the
// 3072 x 4096 first layer of a 4096-wide MLP moves its bytes faster than the
// tile kernel (wgrad_dma_kernel), whose workgroups each load their operand
// tiles, then their master tile, then store it.
//
// LDS (144 KB): two delta chunks [256 b][64 o] bf16, two Wq chunks
// [64 o][64 i] bf16 and the activation strip [256 b][64 i] bf16 (128-byte
// rows), two dW chunks [64 o][64 i] fp32 (256-byte rows).  Batches of at
// most 256 rows (FB_BMAX); backward-weight sums 128 or 256 rows (NKS K16
// steps), zero from row B on.
constexpr int FB_TI = 64, FB_TO = 64, FB_NT = 512, FB_BMAX = 256;
constexpr int FB_NB = 6;  // master chunks a stream thread holds: t - 1 .. t + 4
static_assert(KCHUNK % FB_TO == 0, "chunks of whole o tiles");

// 128-byte-row tiles read both plainly (one 16-byte chunk of 16 consecutive
// rows per 16 lanes) and transposed (ds_read_b64_tr_b16: 4 consecutive rows,
// 4 aligned chunks per 32 lanes).  Chunk c of row r sits at c ^ sw128(r):
// the same-parity rows of 16 consecutive rows take 8 distinct positions, and
// rows 2 apart take opposite halves, so neither read has bank conflicts.
__device__ __forceinline__ int sw128(int r) { return (((r >> 1) & 1) << 2) | ((r >> 2) & 3); }
__device__ __forceinline__ int t128(int r, int c) { return r * 128 + ((c ^ sw128(r)) << 4); }

// MFMA operand from a 128-byte-row tile: 8 consecutive rows (K) of column
// col0 + (lane & 31), rows k0 + 8 (lane >> 5) .. + 7 (see tr_operand).
__device__ __forceinline__ bf16x8 tr128(const char* tile, int k0, int col0, int lane) {
  const int g = lane >> 4, il = lane & 15, a = il & 3, e = il >> 2, h = lane >> 5;
  const int col = col0 + 16 * (g & 1) + 4 * a;
  s16x4 v[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int k = k0 + 8 * h + 4 * q + e;
    v[q] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_s16x4*)(tile + t128(k, col >> 3) + (col & 4) * 2));
  }
  typedef short s16x8 __attribute__((ext_vector_type(8)));
  const s16x8 all = {v[0][0], v[0][1], v[0][2], v[0][3], v[1][0], v[1][1], v[1][2], v[1][3]};
  return __builtin_bit_cast(bf16x8, all);
}
// MFMA operand read plainly: row `row`, 16-byte chunk `c` (8 consecutive K).
__device__ __forceinline__ bf16x8 row128(const char* tile, int row, int c) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(tile + t128(row, c)));
}


// Raw buffer resources (gfx9 descriptor word 3): an access whose byte offset
// is at or beyond `bytes` reads zeros and writes nothing.  Every offset used
// here is a whole 16 / 8 / 4 byte unit inside or outside the range.
constexpr uint32_t kBufWord3 = 0x00020000u;
constexpr uint32_t kOob = 0xFFFFFFF0u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, bytes, kBufWord3);
}

template <bool SPLIT, int NKS, bool DG>
__global__ __launch_bounds__(FB_NT, 1) void bwd_fused_kernel(GemmArgs g, int strips, int nsplit,
                                                             int cps) {
  __shared__ __attribute__((aligned(16))) char smem[144 * 1024 + 2048];
  float* const bpart = reinterpret_cast<float*>(smem + 147456);  // bias block sums [2][4][64]
  auto dbuf = [&](int t) { return smem + (t & 1) * 32768; };                    // delta chunk
  auto wbuf = [&](int t) { return smem + 65536 + (t & 1) * 8192; };             // Wq chunk
  auto wdbuf = [&](int t) { return reinterpret_cast<float*>(smem + 81920 + (t & 1) * 16384); };
  char* const astrip = smem + 114688;  // activation strip [16 NKS][64] bf16

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5;
  const int lin = xcd_work(blockIdx.x, gridDim.x);
  const int per_slot = strips * nsplit;
  const int z = lin / per_slot, rs = lin % per_slot;
  const int split = rs / strips, strip = rs % strips;
  const int I = g.M, B = g.N, O = g.K;
  const int i0 = strip * FB_TI;
  const int nt_all = (O + FB_TO - 1) / FB_TO;
  constexpr int TPC = KCHUNK / FB_TO;
  const int tbeg = SPLIT ? split * cps * TPC : 0;
  const int tend = SPLIT ? (nt_all < tbeg + cps * TPC ? nt_all : tbeg + cps * TPC) : nt_all;
  // steps t = tbeg - 1 .. tend (stream: stage t + 1, update t - 1), padded
  // to whole groups of FB_NB for the stream waves' register rotation
  const int nsteps = (tend - tbeg + 2 + FB_NB - 1) / FB_NB * FB_NB;
  const int Bp = (B + 31) & ~31;  // batch rows of the bias sum; rows B .. Bp - 1 are zero
  // The bias of chunk t belongs to the strip t % strips (spread evenly).
  auto bias_own = [&](int t) { return t % strips == strip; };
  const int nblk = (Bp + 63) / 64;  // 64-row blocks of the bias sum
  static_assert(NKS == 8 || NKS == 16, "batch rows 128 or 256");

  // Activation strip [16 NKS][64] into LDS (all waves), zero from row B and
  // from column I on (a row of the layer-1 input is I wide, unpadded).
  {
    const uint16_t* act = static_cast<const uint16_t*>(g.a) + z * g.a_slot;
#pragma unroll
    for (int p = 0; p < FB_BMAX / 64; ++p) {
      const int row = (tid >> 3) + 64 * p, c = tid & 7;
      const bool in = row < B && i0 + 8 * c < I;
      if (64 * p < 16 * NKS)
        *reinterpret_cast<u32x4*>(astrip + t128(row, c)) =
            load16(in, act + static_cast<int64_t>(in ? row : 0) * g.a_ld + (in ? i0 + 8 * c : 0));
    }
  }
  __syncthreads();

  if (w < 4) {
    // ---------------- stream waves ----------------
    const int rep = g.order[z];
    const int ts = tid;  // 0 .. 255
    const bool refresh = g.wcopy && z < g.wcopy_slots;
    // W_l rows [tbeg * 64, obound) of this workgroup; offsets relative to row
    // tbeg * 64, so rows before it are negative (out of range as unsigned).
    const int row0 = tbeg * FB_TO;
    const int obound = tend * FB_TO < O ? tend * FB_TO : O;
    const uint32_t wbytes = static_cast<uint32_t>(obound - row0) * I * 4;
    const int64_t wbase = g.w_off + static_cast<int64_t>(row0) * I;
    const float* mw_in = g.master_in + static_cast<int64_t>(rep) * g.master_in_slot;
    float* mw = g.master + static_cast<int64_t>(rep) * g.master_slot;
    const __amdgpu_buffer_rsrc_t r_win = buf_rsrc(mw_in + wbase, wbytes);
    const __amdgpu_buffer_rsrc_t r_wout = buf_rsrc(mw + wbase, wbytes);
    const __amdgpu_buffer_rsrc_t r_copy =
        buf_rsrc(refresh ? static_cast<const void*>(g.wcopy + z * g.wcopy_slot + wbase) : mw,
                 refresh ? wbytes / 2 : 0u);
    const uint16_t* dl = static_cast<const uint16_t*>(g.b) + z * g.b_slot;
    const __amdgpu_buffer_rsrc_t r_delta = buf_rsrc(dl, static_cast<uint32_t>(B) * g.b_ld * 2);

    // Byte offsets are a per-thread base (set once) plus a uniform per-chunk
    // term.  A thread outside the strip's columns gets the base 0xC0000000,
    // which no chunk term (|term| < 2^30, W_l under 1 GiB) brings into range;
    // a chunk before tbeg gives a negative term, out of range as unsigned.
    // No memory operation of the loop sits under a branch, so the compiler's
    // counter waits follow the issue order exactly; the bias, which only one
    // strip per chunk updates, is left to a math wave.
    // Master chunk t: thread rows (ts >> 3) + 32 p of the chunk, two pieces
    // h of four columns, i0 + 4 m8 + 32 h .. + 3, so that the 8 lanes of a
    // row load and store whole 128-byte lines of fp32 per instruction.  For
    // the bf16 values (the Wq stage and the copy) each lane pair swaps one
    // piece: lane 2 j + s then holds columns i0 + 8 j + 32 s .. + 7, 16 bytes.
    const int mrow = ts >> 3, m8 = ts & 7, jx = m8 >> 1, sx = m8 & 1;
    constexpr uint32_t kFar = 0xC0000000u;
    uint32_t wbase4[2][2], wbase2[2];
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      // I is a multiple of 8: a piece starting inside the row is whole
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int col = i0 + 4 * m8 + 32 * hh;
        wbase4[p][hh] = col < I ? 4 * static_cast<uint32_t>((mrow + 32 * p) * I + col) : kFar;
      }
      const int col = i0 + 8 * jx + 32 * sx;
      wbase2[p] = col < I ? 2 * static_cast<uint32_t>((mrow + 32 * p) * I + col) : kFar;
    }
    // bf16 of pieces 0 and 1 (two words each) -> the lane's 8 columns
    auto pair_swap = [&](const u32x2& x0, const u32x2& x1) {
      const u32x2 send = sx ? x0 : x1;
      u32x2 recv;
#pragma unroll
      for (int e = 0; e < 2; ++e)  // quad_perm [1, 0, 3, 2]: lane ^ 1
        recv[e] = static_cast<uint32_t>(
            __builtin_amdgcn_mov_dpp(static_cast<int>(send[e]), 0xB1, 0xF, 0xF, true));
      return sx ? u32x4{recv[0], recv[1], x1[0], x1[1]} : u32x4{x0[0], x0[1], recv[0], recv[1]};
    };
    auto pack4 = [](const f32x4& v) {
      return u32x2{f2bf(v[0]) | (f2bf(v[1]) << 16), f2bf(v[2]) | (f2bf(v[3]) << 16)};
    };
    const uint32_t chunk4 = static_cast<uint32_t>(FB_TO * I * 4);  // bytes of 64 fp32 rows
    auto wterm = [&](int t, uint32_t chunk_bytes) {
      return static_cast<uint32_t>(t - tbeg) * chunk_bytes;
    };
    // piece q = 2 p + h: row mrow + 32 p, columns 4 m8 + 32 h .. + 3.  Default
    // cache policy: with the non-temporal one these loads made the launch
    // about 35% slower on some MI355X boxes (the stores stay non-temporal).
    auto master_chunk = [&](int t, int q) {
      return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                           r_win, wbase4[q >> 1][q & 1] + wterm(t, chunk4),
                                           0, 0));
    };
    // Delta chunk t: rows (ts >> 3) + 32 p < 16 NKS, 16-byte chunk ts & 7;
    // zeros beyond the batch (rows out of range) and past the workgroup's
    // chunks (term out of range).
    uint32_t dbase[NKS / 2];
#pragma unroll
    for (int p = 0; p < NKS / 2; ++p)
      dbase[p] = static_cast<uint32_t>(((ts >> 3) + 32 * p) * g.b_ld + 8 * (ts & 7)) * 2;
    // Delta chunk x sits in dreg[(x - tbeg + 1) & 1], master chunk x in
    // mreg[(x - tbeg + 1) % FB_NB].  A load is waited for only by the step
    // that needs it, and memory operations complete in order, so each wait
    // for delta also covers the master rows issued before it: delta three
    // chunks ahead keeps the master loads (four ahead) three steps in flight.
    u32x4 dreg[2][NKS / 2];
    auto load_delta = [&](int t, u32x4 (&dr)[NKS / 2]) {
      const uint32_t term = t < tend ? static_cast<uint32_t>(t) * (FB_TO * 2) : 0x80000000u;
#pragma unroll
      for (int p = 0; p < NKS / 2; ++p)
        dr[p] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(r_delta, dbase[p] + term, 0, 0));
    };

    f32x4 mreg[FB_NB][4];
    // Prologue in the loop's own pattern of memory operations (steps
    // tbeg - 4 .. tbeg - 2: delta t + 3 except at the first, whose chunk is
    // before the range; master t + 4; then the six stores of chunk t - 1,
    // out of range), so that the vector-memory counter state at the loop
    // entry matches the one at its back edge.
#pragma unroll
    for (int v = 0; v < 3; ++v) {
      const int t = tbeg - 4 + v;
      if (v > 0) load_delta(t + 3, dreg[v & 1]);
#pragma unroll
      for (int q = 0; q < 4; ++q) mreg[1 + v][q] = master_chunk(t + 4, q);
#pragma unroll
      for (int p = 0; p < 2; ++p) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
          __builtin_amdgcn_raw_buffer_store_b128(u32x4{0u, 0u, 0u, 0u}, r_wout, kOob, 0, 2);
        __builtin_amdgcn_raw_buffer_store_b128(u32x4{0u, 0u, 0u, 0u}, r_copy, kOob, 0, 2);
      }
    }

    // step t = tbeg - 1 + u
    auto step = [&](int t, auto uc) {
      constexpr int u = decltype(uc)::value;
      constexpr int b_next = (u + 1) % FB_NB, b_ahead = (u + 4) % FB_NB, b_prev = (u + FB_NB - 1) % FB_NB;
      constexpr int d_next = (u + 1) & 1;  // delta of chunks t + 1 and t + 3
      // stage chunk t + 1: delta, and Wq rounded from the master rows
      char* const dt = dbuf(t + 1);
#pragma unroll
      for (int p = 0; p < NKS / 2; ++p)
        *reinterpret_cast<u32x4*>(dt + t128((ts >> 3) + 32 * p, ts & 7)) = dreg[d_next][p];
      if constexpr (DG) {
        char* const wq = wbuf(t + 1);
#pragma unroll
        for (int p = 0; p < 2; ++p)
          *reinterpret_cast<u32x4*>(wq + t128(mrow + 32 * p, jx + 4 * sx)) =
              pair_swap(pack4(mreg[b_next][2 * p]), pack4(mreg[b_next][2 * p + 1]));
      }
      // loads: delta of chunk t + 3, master of chunk t + 4
      load_delta(t + 3, dreg[d_next]);
#pragma unroll
      for (int q = 0; q < 4; ++q) mreg[b_ahead][q] = master_chunk(t + 4, q);
      // update of chunk t - 1 with its dW (rows outside [tbeg, tend) are out
      // of range)
      const float* dws = wdbuf(t - 1);
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const int r = mrow + 32 * p;
        u32x2 cq[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int c = m8 + 8 * h;
          const f32x4 d = *reinterpret_cast<const f32x4*>(dws + r * 64 + ((c ^ (r & 15)) << 2));
          f32x4 wv = mreg[b_prev][2 * p + h];
          for (int e = 0; e < 4; ++e) wv[e] = fmaf(-g.lr, d[e], wv[e]);
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, wv), r_wout,
                                                 wbase4[p][h] + wterm(t - 1, chunk4), 0, 2);
          cq[h] = pack4(wv);
        }
        __builtin_amdgcn_raw_buffer_store_b128(pair_swap(cq[0], cq[1]), r_copy,
                                               wbase2[p] + wterm(t - 1, chunk4 / 2), 0, 2);
      }
      // bias: db[o] = sum_b delta[b][o] in blocks of 64 batch rows, each row
      // by row, block sums left to right.  Stream wave w sums block w of
      // chunk t (column = lane, four rows per transposing read; lane 16 g + j
      // receives column 16 g + j); a math wave adds the blocks one step later.
      if (t >= tbeg && t < tend && bias_own(t)) {
        const char* dtt = dbuf(t);
        const int gq = lane >> 4, a = lane & 3, e = (lane >> 2) & 3;
        const int col = 16 * gq + 4 * a;
        const int r1 = 64 * w + 64 < Bp ? 64 * w + 64 : Bp;
        float part = 0.0f;
        for (int k0 = 64 * w; k0 < r1; k0 += 4) {
          const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_s16x4*)(dtt + t128(k0 + e, col >> 3) + (col & 4) * 2));
#pragma unroll
          for (int q = 0; q < 4; ++q)
            part += __uint_as_float(static_cast<uint32_t>(static_cast<uint16_t>(v[q])) << 16);
        }
        bpart[(t & 1) * 256 + 64 * w + lane] = part;
      }
      __syncthreads();
    };
    for (int u0 = 0; u0 < nsteps; u0 += FB_NB) {
      const int t = tbeg - 1 + u0;
      step(t, Ic<0>());
      step(t + 1, Ic<1>());
      step(t + 2, Ic<2>());
      step(t + 3, Ic<3>());
      step(t + 4, Ic<4>());
      step(t + 5, Ic<5>());
    }
    return;
  }

  // ---------------- math waves ----------------
  const int wb = w - 4;  // 0 .. 3
  f32x16 accd[2][2], tot[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) accd[a][b][r] = tot[a][b][r] = 0.0f;
  const bool dgrad_wave = 64 * wb < B;
  // Bias update by math wave 4 (lane = row of the chunk): the input of chunk
  // t is loaded at step t, the block sums of chunk t - 1 are added at step t.
  const float* b_in = g.master_in + static_cast<int64_t>(g.order[z]) * g.master_in_slot + g.b_off;
  float* b_out = g.master + static_cast<int64_t>(g.order[z]) * g.master_slot + g.b_off;
  float bias_next = 0.0f;
  for (int u = 0; u < nsteps; ++u) {
    const int t = tbeg - 1 + u;
    if (wb == 0) {
      const float bias_cur = bias_next;
      if (t >= tbeg && t < tend && bias_own(t) && t * FB_TO + lane < O)
        bias_next = b_in[t * FB_TO + lane];
      if (t > tbeg && t <= tend && bias_own(t - 1) && (t - 1) * FB_TO + lane < O) {
        const float* bp = bpart + ((t - 1) & 1) * 256;
        float dbias = bp[lane];
        for (int blk = 1; blk < nblk; ++blk) dbias += bp[64 * blk + lane];
        b_out[(t - 1) * FB_TO + lane] = fmaf(-g.lr, dbias, bias_cur);
      }
    }
    if (t >= tbeg && t < tend) {
      const char* dt = dbuf(t);
      const char* wq = wbuf(t);
      // Backward-weight (dW rows o = 32 (wb & 1) .. + 31 of the chunk, input
      // features 32 (wb >> 1) .. + 31): one accumulation chain over the batch,
      // with the four backward-data steps of the chunk (batch rows 64 wb ..
      // + 63, all 64 inputs; waves past the batch compute rows never stored)
      // placed between its links.
      f32x16 accw;
#pragma unroll
      for (int r = 0; r < 16; ++r) accw[r] = 0.0f;
#pragma unroll
      for (int s = 0; s < NKS; ++s) {
        accw = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr128(astrip, 16 * s, 32 * (wb >> 1), lane),
                                                       tr128(dt, 16 * s, 32 * (wb & 1), lane),
                                                       accw, 0, 0, 0);
        if (DG && s % (NKS / 4) == 0) {
          const int k = s / (NKS / 4);
          const bf16x8 a0 = tr128(wq, 16 * k, 0, lane), a1 = tr128(wq, 16 * k, 32, lane);
          const bf16x8 b0 = row128(dt, 64 * wb + (lane & 31), 2 * k + h);
          const bf16x8 b1 = row128(dt, 64 * wb + 32 + (lane & 31), 2 * k + h);
          accd[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, accd[0][0], 0, 0, 0);
          accd[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, accd[0][1], 0, 0, 0);
          accd[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, accd[1][0], 0, 0, 0);
          accd[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, accd[1][1], 0, 0, 0);
        }
      }
      // dW chunk into LDS as [o][i], 16-byte chunk c of row o at c ^ (o & 15)
      float* dws = wdbuf(t);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int o = 32 * (wb & 1) + (lane & 31), c = 8 * (wb >> 1) + 2 * q + h;
        *reinterpret_cast<f32x4*>(dws + o * 64 + ((c ^ (o & 15)) << 2)) =
            f32x4{accw[4 * q], accw[4 * q + 1], accw[4 * q + 2], accw[4 * q + 3]};
      }
      // end of a KCHUNK range of o: chunk sums left to right, or (SPLIT) the
      // chunk's partial
      if (DG && ((t + 1) % TPC == 0 || t + 1 == tend)) {
        if constexpr (SPLIT) {
          if (dgrad_wave) {
            float* part = g.part + z * g.part_slot + static_cast<int64_t>(t / TPC) * B * g.out_ld;
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
              for (int j = 0; j < 2; ++j) {
                const int b = 64 * wb + 32 * j + (lane & 31);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                  const int i = i0 + 32 * a + 8 * q + 4 * h;
                  if (b < B && i < I)
                    *reinterpret_cast<f32x4*>(part + static_cast<int64_t>(b) * g.out_ld + i) =
                        f32x4{accd[a][j][4 * q], accd[a][j][4 * q + 1], accd[a][j][4 * q + 2],
                              accd[a][j][4 * q + 3]};
                }
              }
          }
        } else {
          const bool first = t < TPC;
#pragma unroll
          for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int j = 0; j < 2; ++j) tot[a][j] = first ? accd[a][j] : tot[a][j] + accd[a][j];
        }
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) accd[a][j][r] = 0.0f;
      }
    }
    __syncthreads();
  }

  if (!DG || SPLIT || !dgrad_wave) return;
  // the masks of every group first (loads in flight together; outside the
  // outputs row 0, column 0 is read and not used), then the stores
  f32x4 ea[2][2][4];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int b = 64 * wb + 32 * j + (lane & 31);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = i0 + 32 * a + 8 * q + 4 * h;
        const bool in = b < B && i < I;
        ea[a][j][q] = epi_load<true, GEMM_DGRAD>(g, z, in ? b : 0, in ? i : 0, 4, nullptr);
      }
    }
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int b = 64 * wb + 32 * j + (lane & 31);
      if (b >= B) continue;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = i0 + 32 * a + 8 * q + 4 * h;
        if (i >= I) continue;  // I is a multiple of 8: whole groups of four
        store_out_with<true, GEMM_DGRAD>(g, z, b, i, 4,
                                         f32x4{tot[a][j][4 * q], tot[a][j][4 * q + 1],
                                               tot[a][j][4 * q + 2], tot[a][j][4 * q + 3]},
                                         ea[a][j][q]);
      }
    }
}

// Sum of the split-K partials of slot z in chunk order, then the epilogue.
// One thread per four consecutive rows m..m+3 of column n.
template <bool BF16, int MODE>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs g, int nchunks) {
  const int z = blockIdx.y;
  const int mq = (g.M + 3) / 4;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= static_cast<int64_t>(g.N) * mq) return;
  const int n = static_cast<int>(idx / mq), m = static_cast<int>(idx % mq) * 4;
  const int cnt = (g.M - m >= 4) ? 4 : g.M - m;
  const float* master_in = g.master_in + static_cast<int64_t>(g.order[z]) * g.master_in_slot;
  const f32x4 a = epi_load<BF16, MODE>(g, z, n, m, cnt, master_in);  // issued with the partials
  const float* p = g.part + z * g.part_slot + static_cast<int64_t>(n) * g.out_ld + m;
  const int64_t cs = static_cast<int64_t>(g.N) * g.out_ld;
  f32x4 v;
  if (nchunks <= 4) {
    // all loads first (a chunk past the last reads the last again, unused)
    f32x4 c[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      c[i] = *reinterpret_cast<const f32x4*>(p + static_cast<int64_t>(min(i, nchunks - 1)) * cs);
    v = c[0];
#pragma unroll
    for (int i = 1; i < 4; ++i)
      if (i < nchunks) v = v + c[i];
  } else {
    v = *reinterpret_cast<const f32x4*>(p);
    for (int c = 1; c < nchunks; ++c) v = v + *reinterpret_cast<const f32x4*>(p + c * cs);
  }
  store_out_with<BF16, MODE>(g, z, n, m, cnt, v, a);
}

// One wave per batch row.  NV > 0: the row's C <= 64 NV logits are loaded
// into registers at once (lane l holds columns l, l + 64, ...); NV = 0: any
// C, column loop.  Both sum the exponentials in the same order: each lane
// over its columns left to right, then a butterfly over the lanes.
template <bool BF16_OUT, int NV>
__global__ __launch_bounds__(256) void softmax_ce_kernel(const float* logits, int64_t ld,
                                                         int64_t slot_stride, int C, int B,
                                                         const int32_t* y, const int32_t* gather,
                                                         int64_t gather_slot, void* delta,
                                                         float* loss, int64_t loss_slot,
                                                         int32_t* correct) {
  const int lane = threadIdx.x & 63, z = blockIdx.y;
  const int b = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= B) return;
  const float* row = logits + z * slot_stride + static_cast<int64_t>(b) * ld;
  const int label = y[gather[z * gather_slot + b]];
  const bool label_ok = label >= 0 && label < C;
  const float invB = 1.0f / static_cast<float>(B);
  const int64_t base = z * slot_stride + static_cast<int64_t>(b) * ld;
  auto put = [&](int c, float dv) {
    if constexpr (BF16_OUT)
      static_cast<uint16_t*>(delta)[base + c] = static_cast<uint16_t>(f2bf(dv));
    else
      static_cast<float*>(delta)[base + c] = dv;
  };
  float mx = -INFINITY, s = 0.0f;
  float zl = 0.0f;  // the label's logit
  if constexpr (NV > 0) {
    float v[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) v[k] = lane + 64 * k < C ? row[lane + 64 * k] : -INFINITY;
    // lane label % 64 holds it in v[label / 64]
    float sel = v[0];
#pragma unroll
    for (int k = 1; k < NV; ++k)
      if (k == (label >> 6)) sel = v[k];
    zl = __shfl(sel, label & 63);
#pragma unroll
    for (int k = 0; k < NV; ++k) mx = fmaxf(mx, v[k]);
    for (int d = 32; d >= 1; d >>= 1) mx = fmaxf(mx, __shfl_xor(mx, d));
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      v[k] = lane + 64 * k < C ? expf(v[k] - mx) : 0.0f;
      s += v[k];
    }
    for (int d = 32; d >= 1; d >>= 1) s += __shfl_xor(s, d);
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const int c = lane + 64 * k;
      if (c < C) put(c, (v[k] / s - (c == label ? 1.0f : 0.0f)) * invB);
    }
    for (int c = 64 * NV + lane; c < ld; c += 64) put(c, 0.0f);
    for (int k = 0; k < NV; ++k) {
      const int c = lane + 64 * k;
      if (c >= C && c < ld) put(c, 0.0f);
    }
  } else {
    if (label_ok) zl = row[label];
    for (int c = lane; c < C; c += 64) mx = fmaxf(mx, row[c]);
    for (int d = 32; d >= 1; d >>= 1) mx = fmaxf(mx, __shfl_xor(mx, d));
    for (int c = lane; c < C; c += 64) s += expf(row[c] - mx);
    for (int d = 32; d >= 1; d >>= 1) s += __shfl_xor(s, d);
    for (int c = lane; c < ld; c += 64) {
      float dv = 0.0f;
      if (c < C) dv = (expf(row[c] - mx) / s - (c == label ? 1.0f : 0.0f)) * invB;
      put(c, dv);
    }
  }
  if (lane == 0) {
    loss[z * loss_slot + b] = label_ok ? logf(s) - (zl - mx) : __builtin_nanf("");
    // the label's logit is the largest (ties with another class count)
    if (correct) correct[z * loss_slot + b] = label_ok && zl >= mx ? 1 : 0;
  }
}

__global__ __launch_bounds__(256) void cast_bf16_kernel(const float* master, int64_t master_slot,
                                                        const int32_t* order, uint16_t* wcopy,
                                                        int64_t wcopy_slot, int64_t n) {
  const int z = blockIdx.y;
  const float* src = master + static_cast<int64_t>(order[z]) * master_slot;
  uint16_t* dst = wcopy + z * wcopy_slot;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x * 4;
  for (int64_t i = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) * 4; i < n;
       i += stride) {
    if (i + 4 <= n) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(src + i);
      uint2 o;
      o.x = f2bf(v[0]) | (f2bf(v[1]) << 16);
      o.y = f2bf(v[2]) | (f2bf(v[3]) << 16);
      *reinterpret_cast<uint2*>(dst + i) = o;
    } else {
      for (int64_t e = i; e < n; ++e) dst[e] = static_cast<uint16_t>(f2bf(src[e]));
    }
  }
}

// Evaluation row table: table[z] = 0 for the 64 slot entries, then
// table[64 + i] = i for the n rows.
__global__ __launch_bounds__(256) void eval_rows_kernel(int32_t* table, int64_t n) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n + 64;
       i += stride)
    table[i] = i < 64 ? 0 : static_cast<int32_t>(i - 64);
}

// Summed loss and correct count of n evaluated rows, one workgroup: thread t
// sums the contiguous run of rows [t * run, (t + 1) * run) in row order in
// double (run = ceil(n / 256)); thread 0 adds the 256 run sums left to right.
// Fixed order: the result does not depend on anything but the inputs.
__global__ __launch_bounds__(256) void eval_reduce_kernel(const float* loss, const int32_t* hit,
                                                          int64_t n, double* out_loss,
                                                          int64_t* out_hits) {
  __shared__ double part_loss[256];
  __shared__ int64_t part_hits[256];
  const int t = threadIdx.x;
  const int64_t run = (n + 255) / 256;
  const int64_t r0 = t * run, r1 = r0 + run < n ? r0 + run : n;
  double acc = 0.0;
  int64_t hits = 0;
  for (int64_t i = r0; i < r1; ++i) {
    acc += static_cast<double>(loss[i]);
    hits += hit[i];
  }
  part_loss[t] = acc;
  part_hits[t] = hits;
  __syncthreads();
  if (t == 0) {
    double sum = 0.0;
    int64_t h = 0;
    for (int i = 0; i < 256; ++i) {
      sum += part_loss[i];
      h += part_hits[i];
    }
    *out_loss = sum;
    *out_hits = h;
  }
}

struct AggWeights {
  float w[OSCARS_MAX_K];
};

// Lane group q of a wave (G groups of 64 / G lanes) owns leaves qL .. qL+L-1;
// each lane owns V chunks of four consecutive elements.  The lane sums its
// leaves as a pairwise tree; xor-shuffles over the group bits then join
// neighbouring subtrees, which completes the same balanced tree over
// P = G L leaves.
// Replicas and the global model are streamed once per round: non-temporal.
__device__ __forceinline__ void agg_store(f32x4 v, f32x4* p) { __builtin_nontemporal_store(v, p); }

template <int G, int L, int V>
__global__ __launch_bounds__(256) void aggregate_kernel(float* g, float* reps, AggWeights w,
                                                        int K, int64_t n, int64_t ld, int bcast) {
  constexpr int LPG = 64 / G;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane / LPG, e = lane % LPG;
  const int64_t base = (static_cast<int64_t>(blockIdx.x) * 4 + wave) * (V * LPG * 4);
  f32x4 leaf[V][L];
#pragma unroll
  for (int v = 0; v < V; ++v) {
    const int64_t i0 = base + (v * LPG + e) * 4;
    const int valid = (n - i0 >= 4) ? 4 : static_cast<int>(n - i0 > 0 ? n - i0 : 0);
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const int k = q * L + i;
      f32x4 x = {0.0f, 0.0f, 0.0f, 0.0f};
      if (k < K) {
        const float* p = reps + k * ld + i0;
        if (valid == 4) {
          x = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
        } else {
          for (int t = 0; t < 4; ++t)
            if (t < valid) x[t] = p[t];
        }
        x = x * w.w[k];
      }
      leaf[v][i] = x;
    }
  }
#pragma unroll
  for (int v = 0; v < V; ++v) {
    const int64_t i0 = base + (v * LPG + e) * 4;
    const int valid = (n - i0 >= 4) ? 4 : static_cast<int>(n - i0 > 0 ? n - i0 : 0);
#pragma unroll
    for (int s = 1; s < L; s *= 2)
#pragma unroll
      for (int i = 0; i < L; i += 2 * s) leaf[v][i] = leaf[v][i] + leaf[v][i + s];
    f32x4 r = leaf[v][0];
#pragma unroll
    for (int d = LPG; d < 64; d *= 2) {
      f32x4 o;
#pragma unroll
      for (int t = 0; t < 4; ++t) o[t] = __shfl_xor(r[t], d);
      r = r + o;
    }
    if (valid == 4) {
      if (q == 0) agg_store(r, reinterpret_cast<f32x4*>(g + i0));
      if (bcast) {
#pragma unroll
        for (int i = 0; i < L; ++i) {
          const int k = q * L + i;
          if (k < K) agg_store(r, reinterpret_cast<f32x4*>(reps + k * ld + i0));
        }
      }
    } else if (valid > 0) {
      for (int t = 0; t < valid; ++t) {
        if (q == 0) g[i0 + t] = r[t];
        if (bcast)
          for (int i = 0; i < L; ++i) {
            const int k = q * L + i;
            if (k < K) reps[k * ld + i0 + t] = r[t];
          }
      }
    }
  }
}

// Broadcast of g into every replica, as a write pass of its own.  A
// workgroup copies one piece of g (BC_PIECE elements, two 16-byte chunks per
// thread) into one replica.  Pieces are taken in chunks of BC_CHUNK pieces
// (16 MB of g): all K copies of a chunk are written before the next chunk
// starts, replica after replica.  So the workgroups in flight write long runs
// of one replica (not K interleaved runs of 1 KB each), and each piece of g,
// read K times, is still in the L2 of the XCD that reads it (with BC_CHUNK a
// multiple of 8, every copy of a piece lands on the same XCD).  Measured on
// MI355X for K = 32 x 25.6M after a pass over other memory: 545 against
// 604 us for one 16-byte chunk per thread with the K stores in a row.
// With one replica the pass is a plain copy: copy_kernel, one 16-byte chunk
// per thread (336 against 370 us for 1 GiB).
__global__ __launch_bounds__(256) void copy_kernel(const float* g, float* dst, int64_t n) {
  const int64_t i0 = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (i0 + 4 <= n) {
    agg_store(*reinterpret_cast<const f32x4*>(g + i0), reinterpret_cast<f32x4*>(dst + i0));
  } else {
    for (int64_t i = i0; i < n; ++i) dst[i] = g[i];
  }
}

constexpr int BC_PIECE = 2048;
constexpr int64_t BC_CHUNK = 2048;
__global__ __launch_bounds__(256) void broadcast_kernel(const float* g, float* reps, int K,
                                                        int64_t n, int64_t ld) {
  const int64_t pieces = (n + BC_PIECE - 1) / BC_PIECE;
  const int64_t full = pieces / BC_CHUNK;  // chunks of BC_CHUNK pieces; then a shorter tail
  const int64_t b = blockIdx.x;
  int64_t k, p;
  if (b < full * K * BC_CHUNK) {
    const int64_t c = b / (K * BC_CHUNK), rem = b % (K * BC_CHUNK);
    k = rem / BC_CHUNK;
    p = c * BC_CHUNK + rem % BC_CHUNK;
  } else {
    const int64_t tail = pieces - full * BC_CHUNK, rem = b - full * K * BC_CHUNK;
    k = rem / tail;
    p = full * BC_CHUNK + rem % tail;
  }
  float* dst = reps + k * ld;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int64_t i0 = p * BC_PIECE + j * 1024 + threadIdx.x * 4;
    if (i0 + 4 <= n) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(g + i0);
      agg_store(v, reinterpret_cast<f32x4*>(dst + i0));
    } else {
      for (int64_t i = i0; i < n; ++i) dst[i] = g[i];
    }
  }
}

template <int G, int L, int V>
hipError_t agg_launch(float* g, float* reps, const AggWeights& w, int K, int64_t n, int64_t ld,
                      int bcast, hipStream_t s) {
  constexpr int per_block = 4 * V * (64 / G) * 4;
  const int64_t blocks = (n + per_block - 1) / per_block;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL((aggregate_kernel<G, L, V>), dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     s, g, reps, w, K, n, ld, bcast);
  return hipGetLastError();
}

template <bool BF16, int MODE, int SID, bool SPLIT>
hipError_t gemm_launch_shape(const GemmArgs& g, int n_slots, hipStream_t s) {
  typedef typename ShapeOf<MODE, SID>::type S;
  const int nchunks = SPLIT ? (g.K + KCHUNK - 1) / KCHUNK : 1;
  const int64_t gx =
      static_cast<int64_t>((g.N + S::BN - 1) / S::BN) * ((g.M + S::BM - 1) / S::BM) * nchunks;
  if (gx * n_slots > 0x7FFFFFFF) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(gx), n_slots);
  constexpr bool DMA = SID == SHAPE_W || SID == SHAPE_V;
  static_assert(!DMA || (BF16 && MODE != GEMM_WGRAD), "whole-batch tiles: bf16 forward / backward-data");
  if (g.gather) {
    if constexpr (MODE == GEMM_FWD) {
      if constexpr (DMA)
        hipLaunchKernelGGL((gemm_dma_kernel<MODE, true, SID, SPLIT>), grid, dim3(S::NT), 0, s, g);
      else
        hipLaunchKernelGGL((gemm_kernel<BF16, MODE, true, SID, SPLIT>), grid, dim3(S::NT), 0, s, g);
    } else {
      return hipErrorInvalidValue;  // only the forward pass gathers dataset rows
    }
  } else {
    if constexpr (DMA)
      hipLaunchKernelGGL((gemm_dma_kernel<MODE, false, SID, SPLIT>), grid, dim3(S::NT), 0, s, g);
    else
      hipLaunchKernelGGL((gemm_kernel<BF16, MODE, false, SID, SPLIT>), grid, dim3(S::NT), 0, s, g);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !SPLIT) return e;
  if constexpr (SPLIT) {
    const int64_t work = static_cast<int64_t>(g.N) * ((g.M + 3) / 4);
    hipLaunchKernelGGL((splitk_reduce_kernel<BF16, MODE>),
                       dim3(static_cast<unsigned>((work + 255) / 256), n_slots), dim3(256), 0, s, g,
                       nchunks);
    e = hipGetLastError();
  }
  return e;
}

int device_cu_count() {
  static int cus = 0;
  if (cus == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
      cus = v;
    else
      cus = 256;
  }
  return cus;
}

// Forward / backward-data tilings.  Every tiling sums in the same order, so
// the choice changes only the speed: AUTO tunes each configuration online
// from its own launches and keeps the fastest (gemm_launch).
bool split_fits(const GemmArgs& g, int n_slots) {
  const int nchunks = (g.K + KCHUNK - 1) / KCHUNK;
  const int64_t slot = static_cast<int64_t>(nchunks) * g.N * g.out_ld;
  return nchunks > 1 && g.part && slot * n_slots <= g.part_cap;
}

bool tiling_fits(int t, bool bf16, const GemmArgs& g, int n_slots) {
  switch (t) {
    case GEMM_TILING_L: case GEMM_TILING_M: case GEMM_TILING_S: return true;
    case GEMM_TILING_W: return bf16 && g.N > 128;
    case GEMM_TILING_WS: case GEMM_TILING_VS: return bf16 && g.N > 128 && split_fits(g, n_slots);
    case GEMM_TILING_LS: return split_fits(g, n_slots);
  }
  return false;
}

template <bool BF16, int MODE>
hipError_t launch_tiling(const GemmArgs& g_in, int n_slots, hipStream_t s, int t) {
  if constexpr (BF16) {
    if (t == GEMM_TILING_W) return gemm_launch_shape<true, MODE, SHAPE_W, false>(g_in, n_slots, s);
    if (t == GEMM_TILING_WS || t == GEMM_TILING_VS) {
      GemmArgs g = g_in;
      g.part_slot = static_cast<int64_t>((g.K + KCHUNK - 1) / KCHUNK) * g.N * g.out_ld;
      if (t == GEMM_TILING_WS) return gemm_launch_shape<true, MODE, SHAPE_W, true>(g, n_slots, s);
      return gemm_launch_shape<true, MODE, SHAPE_V, true>(g, n_slots, s);
    }
  }
  if (t == GEMM_TILING_LS) {
    GemmArgs g = g_in;
    g.part_slot = static_cast<int64_t>((g.K + KCHUNK - 1) / KCHUNK) * g.N * g.out_ld;
    return gemm_launch_shape<BF16, MODE, SHAPE_L, true>(g, n_slots, s);
  }
  if (t == GEMM_TILING_M) return gemm_launch_shape<BF16, MODE, SHAPE_M, false>(g_in, n_slots, s);
  if (t == GEMM_TILING_S) return gemm_launch_shape<BF16, MODE, SHAPE_S, false>(g_in, n_slots, s);
  return gemm_launch_shape<BF16, MODE, SHAPE_L, false>(g_in, n_slots, s);
}

// Without timings (stream being captured into a graph): the largest tile
// that still gives every CU a workgroup, split-K when even the smallest
// whole-batch tiles leave CUs idle.
int static_tiling(bool bf16, const GemmArgs& g, int n_slots) {
  const int64_t cus = device_cu_count();
  auto tiles = [&](int bm, int bn) {
    return static_cast<int64_t>((g.M + bm - 1) / bm) * ((g.N + bn - 1) / bn) * n_slots;
  };
  if (bf16 && g.N > 128) {
    if (tiles(128, 256) >= 3 * cus / 4) return GEMM_TILING_W;
    if (tiles(128, 128) >= cus / 2 || !split_fits(g, n_slots)) return GEMM_TILING_L;
    return tiles(64, 256) >= cus / 2 ? GEMM_TILING_WS : GEMM_TILING_VS;
  }
  if (tiles(128, 128) >= cus) return GEMM_TILING_L;
  if (tiles(64, 128) >= cus) return GEMM_TILING_M;
  return GEMM_TILING_S;
}

struct TuneKey {
  int dev, bf16, mode, M, N, K, slots, gather, split;
  bool operator<(const TuneKey& o) const {
    return std::tie(dev, bf16, mode, M, N, K, slots, gather, split) <
           std::tie(o.dev, o.bf16, o.mode, o.M, o.N, o.K, o.slots, o.gather, o.split);
  }
};

constexpr int kTuneRuns = 2;  // timed launches per candidate tiling
struct TuneState {
  struct Timed {
    hipEvent_t ev[2] = {nullptr, nullptr};
    int cand = -1;  // candidate index, -1 when the pair is free
  };
  int cand[GEMM_TILING_COUNT] = {};
  int nc = 0;
  float best_ms[GEMM_TILING_COUNT] = {};
  int runs[GEMM_TILING_COUNT] = {};
  int in_flight[GEMM_TILING_COUNT] = {};
  int choice = -1;
  std::vector<Timed> timed;  // event pairs of timed launches (created on demand)
  // Read every timed launch that has completed.
  hipError_t collect() {
    for (Timed& t : timed) {
      if (t.cand < 0) continue;
      const hipError_t q = hipEventQuery(t.ev[1]);
      if (q == hipErrorNotReady) continue;
      if (q != hipSuccess) return q;
      float ms = 0.0f;
      const hipError_t e = hipEventElapsedTime(&ms, t.ev[0], t.ev[1]);
      if (e != hipSuccess) return e;
      const int c = t.cand;
      if (runs[c] == 0 || ms < best_ms[c]) best_ms[c] = ms;
      ++runs[c];
      --in_flight[c];
      t.cand = -1;
    }
    return hipSuccess;
  }
  hipError_t free_slot(Timed** out) {
    for (Timed& t : timed)
      if (t.cand < 0) {
        *out = &t;
        return hipSuccess;
      }
    Timed t;
    hipError_t e = hipEventCreate(&t.ev[0]);
    if (e == hipSuccess) e = hipEventCreate(&t.ev[1]);
    if (e != hipSuccess) return e;
    timed.push_back(t);
    *out = &timed.back();
    return hipSuccess;
  }
};
thread_local bool t_tune_now = false;  // set_gemm_tune_now

}  // namespace

// The tiling state of one context: a forced tiling, or per configuration
// (device, precision, mode, shape, active replicas, gather, split) the online
// tuning and its choice.
struct GemmTuner {
  std::mutex mu;
  int forced = GEMM_TILING_AUTO;
  std::map<TuneKey, TuneState> map;
  ~GemmTuner() {
    for (auto& kv : map)
      for (TuneState::Timed& t : kv.second.timed)
        for (hipEvent_t e : t.ev)
          if (e) (void)hipEventDestroy(e);
  }
};

namespace {

// tuner == nullptr, or tune == false: no timing, no events; a configuration
// the tuner has decided keeps its choice, any other takes the fixed rule.
template <bool BF16, int MODE>
hipError_t gemm_launch(const GemmArgs& g, int n_slots, hipStream_t s, GemmTuner* tuner,
                       bool tune) {
  if constexpr (MODE == GEMM_WGRAD) {
    if constexpr (BF16) {
      const int64_t gx = static_cast<int64_t>((g.M + 127) / 128) * ((g.N + 127) / 128);
      if (gx * n_slots > 0x7FFFFFFF) return hipErrorInvalidValue;
      hipLaunchKernelGGL((wgrad_dma_kernel<WGRAD_MIN_WAVES, WGRAD_PRE>), dim3(static_cast<unsigned>(gx), n_slots),
                         dim3(256), 0, s, g);
      return hipGetLastError();
    }
    return gemm_launch_shape<BF16, MODE, SHAPE_L, false>(g, n_slots, s);
  } else {
    if (!tuner) return launch_tiling<BF16, MODE>(g, n_slots, s, static_tiling(BF16, g, n_slots));
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) dev = 0;
    const TuneKey key{dev, BF16, MODE, g.M, g.N, g.K, n_slots, g.gather != nullptr,
                      split_fits(g, n_slots)};
    std::lock_guard<std::mutex> lock(tuner->mu);
    const int forced = tuner->forced;
    if (forced != GEMM_TILING_AUTO) {
      int t = forced;
      if (!tiling_fits(t, BF16, g, n_slots))
        t = (t == GEMM_TILING_W || t == GEMM_TILING_LS || !BF16 || g.N <= 128) ? GEMM_TILING_L
                                                                                : GEMM_TILING_W;
      return launch_tiling<BF16, MODE>(g, n_slots, s, t);
    }
    if (!tune) {
      const auto it = tuner->map.find(key);
      const int t = it != tuner->map.end() && it->second.choice >= 0
                        ? it->second.choice : static_tiling(BF16, g, n_slots);
      return launch_tiling<BF16, MODE>(g, n_slots, s, t);
    }
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cap) != hipSuccess || cap != hipStreamCaptureStatusNone)
      return launch_tiling<BF16, MODE>(g, n_slots, s, static_tiling(BF16, g, n_slots));

    // Online choice: while a configuration is being tuned, each of its launches
    // runs one candidate tiling between two events (the launches of the real
    // workload, so caches are as warm or cold as they will be); completed
    // event pairs are read at later launches without waiting.  Once every
    // candidate has kTuneRuns timed launches, the one with the smallest time
    // (its fastest launch) is kept.
    TuneState& ts = tuner->map[key];
    if (ts.choice >= 0) return launch_tiling<BF16, MODE>(g, n_slots, s, ts.choice);
    if (ts.nc == 0) {
      for (int t = GEMM_TILING_L; t < GEMM_TILING_COUNT; ++t)
        if (tiling_fits(t, BF16, g, n_slots)) ts.cand[ts.nc++] = t;
      if (ts.nc == 1) ts.choice = ts.cand[0];
      if (ts.nc <= 1) return launch_tiling<BF16, MODE>(g, n_slots, s, ts.cand[0]);
    }
    hipError_t e = ts.collect();
    if (e != hipSuccess) return e;
    if (t_tune_now) {
      // Decided at once: every candidate computes the (identical) result
      // three times, timed; its time is the faster of the last two runs.
      TuneState::Timed* slot = nullptr;
      e = ts.free_slot(&slot);
      float best_ms = 0.0f;
      for (int c = 0; c < ts.nc && e == hipSuccess; ++c) {
        float t_best = 0.0f;
        for (int rep = 0; rep < 3 && e == hipSuccess; ++rep) {
          float ms = 0.0f;
          e = hipEventRecord(slot->ev[0], s);
          if (e == hipSuccess) e = launch_tiling<BF16, MODE>(g, n_slots, s, ts.cand[c]);
          if (e == hipSuccess) e = hipEventRecord(slot->ev[1], s);
          if (e == hipSuccess) e = hipEventSynchronize(slot->ev[1]);
          if (e == hipSuccess) e = hipEventElapsedTime(&ms, slot->ev[0], slot->ev[1]);
          if (rep == 1 || (rep == 2 && ms < t_best)) t_best = ms;
        }
        if (e == hipSuccess && (c == 0 || t_best < best_ms)) {
          best_ms = t_best;
          ts.choice = ts.cand[c];
        }
      }
      return e;  // the result is in place (every timed run computed it)
    }
    int next = -1;
    bool done = true;
    for (int c = 0; c < ts.nc; ++c) {
      if (ts.runs[c] + ts.in_flight[c] < kTuneRuns && (next < 0 || ts.runs[c] + ts.in_flight[c] <
                                                                     ts.runs[next] + ts.in_flight[next]))
        next = c;
      if (ts.runs[c] < kTuneRuns) done = false;
    }
    if (done) {
      int c_best = 0;
      for (int c = 1; c < ts.nc; ++c)
        if (ts.best_ms[c] < ts.best_ms[c_best]) c_best = c;
      ts.choice = ts.cand[c_best];
      return launch_tiling<BF16, MODE>(g, n_slots, s, ts.choice);
    }
    if (next < 0)  // every remaining run is in flight: launch the provisional choice
      return launch_tiling<BF16, MODE>(g, n_slots, s, static_tiling(BF16, g, n_slots));
    TuneState::Timed* slot = nullptr;
    e = ts.free_slot(&slot);
    if (e != hipSuccess) return e;
    e = hipEventRecord(slot->ev[0], s);
    if (e == hipSuccess) e = launch_tiling<BF16, MODE>(g, n_slots, s, ts.cand[next]);
    if (e == hipSuccess) e = hipEventRecord(slot->ev[1], s);
    if (e != hipSuccess) return e;
    slot->cand = next;
    ++ts.in_flight[next];
    return hipSuccess;
  }
}

}  // namespace

GemmTuner* gemm_tuner_create() { return new (std::nothrow) GemmTuner(); }

void gemm_tuner_destroy(GemmTuner* t) { delete t; }

void gemm_tuner_set_tiling(GemmTuner* tuner, int tiling) {
  std::lock_guard<std::mutex> lock(tuner->mu);
  tuner->forced = tiling;
  // AUTO starts over: every configuration is tuned again at its next launches
  // (event pairs still in flight are left to complete and are not read).
  for (auto& kv : tuner->map) {
    TuneState& ts = kv.second;
    ts.nc = 0;
    ts.choice = -1;
    for (int c = 0; c < GEMM_TILING_COUNT; ++c) ts.runs[c] = ts.in_flight[c] = 0;
    for (TuneState::Timed& t : ts.timed) t.cand = -1;
  }
}

void set_gemm_tune_now(bool on) { t_tune_now = on; }

int gemm_tuner_pending(GemmTuner* tuner) {
  std::lock_guard<std::mutex> lock(tuner->mu);
  int n = 0;
  for (const auto& kv : tuner->map) n += kv.second.nc > 0 && kv.second.choice < 0;  // launched, undecided
  return n;
}

hipError_t launch_gemm(const GemmArgs& g, GemmMode mode, bool bf16, int n_slots, hipStream_t s,
                       GemmTuner* tuner, bool tune) {
  if (bf16) {
    switch (mode) {
      case GEMM_FWD: return gemm_launch<true, GEMM_FWD>(g, n_slots, s, tuner, tune);
      case GEMM_DGRAD: return gemm_launch<true, GEMM_DGRAD>(g, n_slots, s, tuner, tune);
      case GEMM_WGRAD: return gemm_launch<true, GEMM_WGRAD>(g, n_slots, s, tuner, tune);
    }
  } else {
    switch (mode) {
      case GEMM_FWD: return gemm_launch<false, GEMM_FWD>(g, n_slots, s, tuner, tune);
      case GEMM_DGRAD: return gemm_launch<false, GEMM_DGRAD>(g, n_slots, s, tuner, tune);
      case GEMM_WGRAD: return gemm_launch<false, GEMM_WGRAD>(g, n_slots, s, tuner, tune);
    }
  }
  return hipErrorInvalidValue;
}

// Batches of at most FB_BMAX rows, whole 16-byte input chunks, and W_l (with
// the chunks read ahead) under 1 GiB, so that 32-bit buffer offsets with an
// out-of-range base never wrap into range.
bool backward_fusable(const GemmArgs& g) {
  return g.N >= 1 && g.N <= FB_BMAX && g.M % 8 == 0 &&
         static_cast<int64_t>(g.K + 6 * FB_TO) * g.M * 4 < (static_cast<int64_t>(1) << 30);
}

bool backward_fused_enabled(int mode) { return mode != BACKWARD_SEPARATE; }

// Grid x = slots x strips x splits, slot slowest, strip fastest: with the
// XCD-aware order the strips of one slot (which read the same delta) share
// an XCD and its L2.  A workgroup covers `cps` chunks of KCHUNK output
// features (all of them: no split).  Without a forced mode cps (all chunks,
// or ..., 4, 2, 1) is the one whose workgroups fill their last pass over the
// CUs best, the largest on ties (a split costs partial traffic and a
// reduce); measured on MI355X against the other choices at 1 to 8 replicas
// of 4096 x 4096 layers.
int bwd_fused_splits(const GemmArgs& g, int n_slots, int* cps, int max, bool dgrad) {
  if (!backward_fusable(g) || n_slots < 1 || max < 1) return 0;
  const int nchunks = (g.K + KCHUNK - 1) / KCHUNK;
  const int64_t part_slot = static_cast<int64_t>(nchunks) * g.N * g.out_ld;
  const bool can_split =
      nchunks > 1 && (!dgrad || (g.part && part_slot * n_slots <= g.part_cap));
  int n = 0;
  for (int c = nchunks; n < max; c = (c + 1) / 2) {
    cps[n++] = c;
    if (c == 1 || !can_split) break;
  }
  return n;
}

hipError_t launch_bwd_fused(const GemmArgs& g_in, int n_slots, hipStream_t s, int mode,
                            int cps_forced, bool dgrad) {
  if (!backward_fusable(g_in) || n_slots < 1) return hipErrorInvalidValue;
  GemmArgs g = g_in;
  const int strips = (g.M + FB_TI - 1) / FB_TI;
  const int nchunks = (g.K + KCHUNK - 1) / KCHUNK;
  g.part_slot = dgrad ? static_cast<int64_t>(nchunks) * g.N * g.out_ld : 0;
  const bool can_split =
      nchunks > 1 && (!dgrad || (g.part && g.part_slot * n_slots <= g.part_cap));
  int cps = nchunks;
  if (cps_forced > 0) {
    cps = can_split && cps_forced < nchunks ? cps_forced : nchunks;
  } else if (can_split && mode == BACKWARD_FUSED_SPLIT) {
    cps = 1;
  } else if (can_split && mode == BACKWARD_AUTO) {
    const int64_t cus = device_cu_count();
    double best = -1.0;
    for (int c = nchunks;; c = (c + 1) / 2) {
      const int64_t wgs = static_cast<int64_t>(n_slots) * strips * ((nchunks + c - 1) / c);
      const double fill = static_cast<double>(wgs) / static_cast<double>((wgs + cus - 1) / cus * cus);
      if (fill > best + 1e-9) {
        best = fill;
        cps = c;
      }
      if (c == 1) break;
    }
  }
  const bool split = cps < nchunks;
  const int nsplit = (nchunks + cps - 1) / cps;
  const int64_t gx = static_cast<int64_t>(n_slots) * strips * nsplit;
  if (gx > 0x7FFFFFFF) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(gx)), block(FB_NT);
  const bool b256 = g.N > 128;  // batch rows summed by backward-weight: 256 or 128
  if (!dgrad) {  // update only: a split range is a workgroup's own (no partials)
    if (b256) hipLaunchKernelGGL((bwd_fused_kernel<true, 16, false>), grid, block, 0, s, g, strips, nsplit, cps);
    else hipLaunchKernelGGL((bwd_fused_kernel<true, 8, false>), grid, block, 0, s, g, strips, nsplit, cps);
    return hipGetLastError();
  }
  if (!split) {
    if (b256) hipLaunchKernelGGL((bwd_fused_kernel<false, 16, true>), grid, block, 0, s, g, strips, 1, cps);
    else hipLaunchKernelGGL((bwd_fused_kernel<false, 8, true>), grid, block, 0, s, g, strips, 1, cps);
    return hipGetLastError();
  }
  if (b256) hipLaunchKernelGGL((bwd_fused_kernel<true, 16, true>), grid, block, 0, s, g, strips, nsplit, cps);
  else hipLaunchKernelGGL((bwd_fused_kernel<true, 8, true>), grid, block, 0, s, g, strips, nsplit, cps);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t work = static_cast<int64_t>(g.N) * ((g.M + 3) / 4);
  hipLaunchKernelGGL((splitk_reduce_kernel<true, GEMM_DGRAD>),
                     dim3(static_cast<unsigned>((work + 255) / 256), n_slots), dim3(256), 0, s, g,
                     nchunks);
  return hipGetLastError();
}

template <bool BF16_OUT, int NV>
void softmax_launch(const float* logits, int64_t ld, int64_t slot_stride, int C, int B,
                    const int32_t* y, const int32_t* gather, int64_t gather_slot, void* delta,
                    float* loss, int64_t loss_slot, int n_slots, hipStream_t s, int32_t* correct) {
  hipLaunchKernelGGL((softmax_ce_kernel<BF16_OUT, NV>), dim3((B + 3) / 4, n_slots), dim3(256), 0, s,
                     logits, ld, slot_stride, C, B, y, gather, gather_slot, delta, loss, loss_slot,
                     correct);
}

template <bool BF16_OUT>
void softmax_dispatch(const float* logits, int64_t ld, int64_t slot_stride, int C, int B,
                      const int32_t* y, const int32_t* gather, int64_t gather_slot, void* delta,
                      float* loss, int64_t loss_slot, int n_slots, hipStream_t s, int32_t* correct) {
  const int nv = (C + 63) / 64;
  if (nv <= 1)
    softmax_launch<BF16_OUT, 1>(logits, ld, slot_stride, C, B, y, gather, gather_slot, delta, loss,
                                loss_slot, n_slots, s, correct);
  else if (nv <= 4)
    softmax_launch<BF16_OUT, 4>(logits, ld, slot_stride, C, B, y, gather, gather_slot, delta, loss,
                                loss_slot, n_slots, s, correct);
  else if (nv <= 16)
    softmax_launch<BF16_OUT, 16>(logits, ld, slot_stride, C, B, y, gather, gather_slot, delta, loss,
                                 loss_slot, n_slots, s, correct);
  else
    softmax_launch<BF16_OUT, 0>(logits, ld, slot_stride, C, B, y, gather, gather_slot, delta, loss,
                                loss_slot, n_slots, s, correct);
}

hipError_t launch_softmax_ce(const float* logits, int64_t ld, int64_t slot_stride, int C, int B,
                             const int32_t* y, const int32_t* gather, int64_t gather_slot,
                             void* delta, bool delta_bf16, float* loss, int64_t loss_slot,
                             int n_slots, hipStream_t s, int32_t* correct) {
  if (B < 1 || n_slots < 1) return hipSuccess;
  if (delta_bf16)
    softmax_dispatch<true>(logits, ld, slot_stride, C, B, y, gather, gather_slot, delta, loss,
                           loss_slot, n_slots, s, correct);
  else
    softmax_dispatch<false>(logits, ld, slot_stride, C, B, y, gather, gather_slot, delta, loss,
                            loss_slot, n_slots, s, correct);
  return hipGetLastError();
}

hipError_t launch_cast_bf16(const float* master, int64_t master_slot, const int32_t* order,
                            uint16_t* wcopy, int64_t wcopy_slot, int64_t n, int n_slots,
                            hipStream_t s) {
  int64_t blocks = (n / 4 + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(cast_bf16_kernel, dim3(static_cast<unsigned>(blocks), n_slots), dim3(256), 0,
                     s, master, master_slot, order, wcopy, wcopy_slot, n);
  return hipGetLastError();
}

hipError_t launch_eval_rows(int32_t* table, int64_t n, hipStream_t s) {
  int64_t blocks = (n + 64 + 255) / 256;
  if (blocks > 2048) blocks = 2048;
  hipLaunchKernelGGL(eval_rows_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, table,
                     n);
  return hipGetLastError();
}

hipError_t launch_eval_reduce(const float* loss, const int32_t* hit, int64_t n, double* out_loss,
                              int64_t* out_hits, hipStream_t s) {
  hipLaunchKernelGGL(eval_reduce_kernel, dim3(1), dim3(256), 0, s, loss, hit, n, out_loss,
                     out_hits);
  return hipGetLastError();
}

// Leaves per lane and lane groups: P = G L with at most 4 groups of 16 lanes
// (measured best on MI355X for K = 8, 16, 32 against 1, 2 and 8 groups and
// two chunks per lane).
constexpr int AGG_GMAX = 4, AGG_V = 1;
// From this many replicas on the broadcast is a pass of its own (K = 32:
// 5.5 -> 5.8 TB/s on MI355X; K = 8 is faster fused).
constexpr int AGG_SPLIT_K = 16;
template <int P>
hipError_t agg_dispatch(float* g, float* reps, const AggWeights& w, int K, int64_t n, int64_t ld,
                        int bcast, hipStream_t s) {
  constexpr int G = P < AGG_GMAX ? P : AGG_GMAX;
  // From AGG_SPLIT_K replicas on, the broadcast runs as its own pass:
  // HBM then sees a read phase and a write phase instead of K + 1 interleaved
  // write streams per workgroup.  The values written are the same.
  if (!bcast || K < AGG_SPLIT_K)
    return agg_launch<G, P / G, AGG_V>(g, reps, w, K, n, ld, bcast, s);
  hipError_t e = agg_launch<G, P / G, AGG_V>(g, reps, w, K, n, ld, 0, s);
  if (e != hipSuccess) return e;
  return launch_broadcast(g, reps, K, n, ld, s);
}

hipError_t launch_broadcast(const float* g, float* replicas, int K, int64_t n, int64_t ld,
                            hipStream_t s) {
  if (K == 1) {
    const int64_t blocks = (n + 1023) / 1024;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(copy_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, g,
                       replicas, n);
    return hipGetLastError();
  }
  const int64_t blocks = (n + BC_PIECE - 1) / BC_PIECE * K;
  if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(broadcast_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, g,
                     replicas, K, n, ld);
  return hipGetLastError();
}

hipError_t launch_aggregate(float* g, float* replicas, const float* w, int K, int64_t n,
                            int64_t ld, int broadcast, hipStream_t s) {
  AggWeights aw;
  for (int k = 0; k < OSCARS_MAX_K; ++k) aw.w[k] = k < K ? w[k] : 0.0f;
  int P = 1;
  while (P < K) P *= 2;
  switch (P) {
    case 1: return agg_dispatch<1>(g, replicas, aw, K, n, ld, broadcast, s);
    case 2: return agg_dispatch<2>(g, replicas, aw, K, n, ld, broadcast, s);
    case 4: return agg_dispatch<4>(g, replicas, aw, K, n, ld, broadcast, s);
    case 8: return agg_dispatch<8>(g, replicas, aw, K, n, ld, broadcast, s);
    case 16: return agg_dispatch<16>(g, replicas, aw, K, n, ld, broadcast, s);
    case 32: return agg_dispatch<32>(g, replicas, aw, K, n, ld, broadcast, s);
    case 64: return agg_dispatch<64>(g, replicas, aw, K, n, ld, broadcast, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace oscars
