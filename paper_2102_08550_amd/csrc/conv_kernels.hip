// Device code of the convolutional workload for gfx950 (CDNA4), fp32.
//
// Every pass is one implicit GEMM C[m][n] = sum_k A(m, k) B(n, k) whose
// operands are gathered on the fly (no im2col matrix in HBM):
//
//   pass        M               N              K              A(m, k)              B(n, k)
//   CONV_FWD    output pixels   Cout           9 Cin          input tap            W[n][k]
//   CONV_DGRAD  input pixels    Cin            9 Cout         output-gradient tap  W[o][r][s][n]
//   CONV_WGRAD  Cout            9 Cin + 1      output pixels  dZ[k][m]             input tap (1 for
//                                                                                  the bias column)
//   FC_FWD      batch           classes        channels       pooled[m][k]         W[n][k]
//   FC_DGRAD    batch           channels       classes        delta[m][k]          W[k][n]
//   FC_WGRAD    classes         channels + 1   batch          delta[k][m]          pooled[k][n] (1)
//
// with k = (r 3 + s) Cin + c for the conv taps (the layout of W[o][3][3][c]).
// Backward-data of a stride-2 layer treats each parity class of the input
// pixels as a GEMM of its own: input row hi receives output row i through tap
// r only where hi + 1 - r = 2 i, so even rows take tap r = 1 and odd rows taps
// 0 and 2 (likewise columns).  Each class gathers only its 1, 2 or 4 taps
// (K = taps x Cout), a quarter of the 9-tap work on average; the four classes
// share one launch (their tiles concatenated, the most taps first).
// A workgroup computes a 64 x 64 tile of C with four waves of 32 x 32, fp32
// MFMA 32x32x2, K in steps of 16: later steps' operands are gathered into
// registers while the current step's MFMAs read LDS (two LDS buffers, one
// barrier per step; two register sets where the channel counts allow loaders
// without branches).  Where one side of the GEMM is at most 32 channels
// (backward-data into, forward into, or backward-weight of 32 channels or
// fewer) 128 x 32 or 32 x 128 tiles take its place, and layers with at most three input channels (layer 1) have a
// direct forward and a one-accumulator backward-weight of their own.  The
// weight-gradient passes split K into ranges, one partial sum per range,
// which the update kernel adds in a fixed order (eight groups of consecutive
// ranges) before applying the SGD step of Eq. 4 -- so results depend on
// nothing but the inputs, whichever slots share a launch.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "conv.h"

namespace oscars {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

// A compile-time integer passed as an argument (static register indices).
template <int U> struct Pi { static constexpr int value = U; };

// Schedule of a K step with N MFMAs: each MFMA followed by a share of the
// step's other work (its next operands' LDS reads, gather address
// arithmetic, LDS stores, global loads), which then issues while the matrix
// core runs.  Without it the compiler issued the MFMAs back to back and the
// rest after them; with one or two waves per SIMD (one or two replicas)
// nothing else hid that work.
template <int N>
__device__ __forceinline__ void interleave() {
#pragma unroll
  for (int u = 0; u < N; ++u) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // LDS reads
    __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);  // VALU
    __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // LDS write
    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // global load
  }
}

constexpr int CT = 64;       // tile rows and columns
constexpr int CK = 16;       // K per step
constexpr int CLD = CT + 4;  // LDS row pitch (floats)

struct Dims {
  int64_t M, N, K;
};

// Loads never sit behind a branch in the vector loaders: a lane with nothing
// to load (padding, a row or K past the end) reads these zeros instead, so
// that the compiler's memory-counter waits stay exact and a load of the next
// K steps can stay in flight across a wait for the current one.
__device__ __attribute__((aligned(16))) float k_conv_zero[4];
// and ones for the bias column of a weight gradient
__device__ __attribute__((aligned(16))) float k_conv_one[4] = {1.0f, 1.0f, 1.0f, 1.0f};

// Stride-2 backward-data class `cls`: input rows hi = 2 i + (cls >> 1), columns
// wi = 2 j + (cls & 1); per dimension one tap (r = 1) for even, two (r = 0, 2)
// for odd positions.
__host__ __device__ inline int cls_rows(const ConvArgs& a) { return (a.H - (a.cls >> 1) + 1) / 2; }
__host__ __device__ inline int cls_cols(const ConvArgs& a) { return (a.W - (a.cls & 1) + 1) / 2; }
__host__ __device__ inline int cls_taps(int odd) { return odd ? 2 : 1; }

__host__ __device__ inline Dims pass_dims(const ConvArgs& a, int pass) {
  switch (pass) {
    case CONV_FWD: return {static_cast<int64_t>(a.B) * a.Ho * a.Wo, a.Co, 9LL * a.C};
    case CONV_DGRAD:
      if (a.stride == 2)
        return {static_cast<int64_t>(a.B) * cls_rows(a) * cls_cols(a), a.C,
                static_cast<int64_t>(cls_taps(a.cls >> 1)) * cls_taps(a.cls & 1) * a.Co};
      return {static_cast<int64_t>(a.B) * a.H * a.W, a.C, 9LL * a.Co};
    case CONV_WGRAD: return {a.Co, 9LL * a.C + 1, static_cast<int64_t>(a.B) * a.Ho * a.Wo};
    case FC_FWD: return {a.B, a.Co, a.C};
    case FC_DGRAD: return {a.B, a.C, a.Co};
    default: return {a.Co, static_cast<int64_t>(a.C) + 1, a.B};  // FC_WGRAD
  }
}

typedef float f32x4 __attribute__((ext_vector_type(4)));

// Kernel tap (r, s) of backward-data tap index t: all nine (t = 3 r + s) for
// stride 1; the class's one, two or four for stride 2.
__device__ __forceinline__ void dgrad_tap(const ConvArgs& a, int t, int& r, int& s) {
  if (a.stride == 2) {
    const int oc = a.cls & 1, tr = t >> oc, ts = t - (tr << oc);  // cls_taps(oc) = 1 << oc
    r = (a.cls >> 1) ? 2 * tr : 1;
    s = oc ? 2 * ts : 1;
  } else {
    r = t / 3;
    s = t - 3 * r;
  }
}

// A thread's K sequence k0, k0 + CK, k0 + 2 CK, ... (or another step) split
// as k = q D + r: one division when constructed, then next() steps without
// dividing (step = dq D + dr, split once).
struct KCursor {
  int q, r, D, dq, dr;
  __device__ KCursor() = default;
  __device__ KCursor(int k0, int D_, int step = CK) : D(D_) {
    q = k0 / D;
    r = k0 - q * D;
    dq = step / D;
    dr = step - dq * D;
  }
  __device__ __forceinline__ void next() {
    r += dr;
    q += dq;
    const bool w = r >= D;
    r = w ? r - D : r;
    q = w ? q + 1 : q;
  }
};

// The same for an output pixel k = (b Ho + i) Wo + j: a step of `step`
// pixels is db whole images and a remainder of di rows and dj columns, so
// that each coordinate wraps at most once per step (no loop, no branch).
struct PixCursor {
  int b, i, j, Ho, Wo, db, di, dj;
  __device__ PixCursor() = default;
  __device__ PixCursor(int k0, int Ho_, int Wo_, int step = CK) : Ho(Ho_), Wo(Wo_) {
    const int hw = Ho * Wo;
    b = k0 / hw;
    const int p = k0 - b * hw;
    i = p / Wo;
    j = p - i * Wo;
    db = step / hw;
    const int rest = step - db * hw;
    di = rest / Wo;
    dj = rest - di * Wo;
  }
  __device__ __forceinline__ void next() {
    j += dj;
    i += di;
    b += db;
    const bool wj = j >= Wo;
    j = wj ? j - Wo : j;
    i = wj ? i + 1 : i;
    const bool wi = i >= Ho;
    i = wi ? i - Ho : i;
    b = wi ? b + 1 : b;
  }
};

// Input pixels of consecutive backward-data rows (the class's pixel grid for
// stride 2, the image for stride 1): decoded once, then stepped forward.
struct DgradRowWalker {
  const ConvArgs& a;
  int b, i, j, rows, cols;
  __device__ DgradRowWalker(const ConvArgs& a_, int m) : a(a_) {
    rows = a.stride == 2 ? cls_rows(a) : a.H;
    cols = a.stride == 2 ? cls_cols(a) : a.W;
    const int hw = rows * cols;
    b = m / hw;
    const int p = m - b * hw;
    i = p / cols;
    j = p - i * cols;
  }
  __device__ __forceinline__ void advance(int d) {
    j += d;
    while (j >= cols) {
      j -= cols;
      if (++i == rows) {
        i = 0;
        ++b;
      }
    }
  }
  // offset of channel 0 of the pixel in [B][H][W][C]
  __device__ __forceinline__ int64_t offset() const {
    const int hi = a.stride == 2 ? 2 * i + (a.cls >> 1) : i;
    const int wi = a.stride == 2 ? 2 * j + (a.cls & 1) : j;
    return ((static_cast<int64_t>(b) * a.H + hi) * a.W + wi) * a.C;
  }
};

// Loaders.  A thread gathers, per K step, four consecutive K elements of one
// A row (m0 + t / 4) and of one B row (n0 + t / 4).  What depends only on
// the row (the pixel's image and position, or the weight tap of a column) is
// decoded once per workgroup; the K index is decoded once per step and
// stepped through the four elements.  Where the four elements are
// consecutive channels of one tap (channel counts a multiple of 4) they are
// one 16-byte load.  Sizes fit 32-bit indices (oscars_create_cnn checks).
template <int PASS>
struct ConvLoader {
  const ConvArgs& a;
  int kend;
  // A row
  bool am = false;
  const float* arow = nullptr;
  int ah = 0, aw = 0;
  int am_idx = 0;
  // B row
  bool bn = false, bones = false;
  int bn_idx = 0, br = 0, bs = 0, bc = 0;
  const float* in = nullptr;
  const int32_t* rows = nullptr;
  const float* dz = nullptr;
  const float* Wt = nullptr;

  __device__ ConvLoader(const ConvArgs& a_, int kend_, int m, int M, int n, int N, const float* in_,
                        const int32_t* rows_, const float* dz_, const float* Wt_)
      : a(a_), kend(kend_), am(m < M), am_idx(m), bn(n < N), bn_idx(n), in(in_), rows(rows_),
        dz(dz_), Wt(Wt_) {
    if constexpr (PASS == CONV_FWD) {
      if (am) {
        const int hw = a.Ho * a.Wo, b = m / hw, p = m - b * hw, i = p / a.Wo, j = p - i * a.Wo;
        arow = image(b);
        ah = a.stride * i - 1;
        aw = a.stride * j - 1;
      }
    } else if constexpr (PASS == CONV_DGRAD) {
      if (am) {
        int b, hi, wi;
        dgrad_pixel(a, m, b, hi, wi);
        arow = dz + static_cast<int64_t>(b) * a.Ho * a.Wo * a.Co;
        ah = hi + 1;
        aw = wi + 1;
      }
    } else if constexpr (PASS == CONV_WGRAD) {
      if (bn) {
        bones = n == 9 * a.C;
        if (!bones) {
          const int rs = n / a.C;
          bc = n - rs * a.C;
          br = rs / 3;
          bs = rs - 3 * br;
        }
      }
    }
  }

  // Input pixel (b, hi, wi) of backward-data row m.
  static __device__ __forceinline__ void dgrad_pixel(const ConvArgs& a, int m, int& b, int& hi,
                                                     int& wi) {
    if (a.stride == 2) {
      const int rows = cls_rows(a), cols = cls_cols(a), hw = rows * cols;
      b = m / hw;
      const int p = m - b * hw, i = p / cols;
      hi = 2 * i + (a.cls >> 1);
      wi = 2 * (p - i * cols) + (a.cls & 1);
    } else {
      const int hw = a.H * a.W;
      b = m / hw;
      const int p = m - b * hw;
      hi = p / a.W;
      wi = p - hi * a.W;
    }
  }

  __device__ __forceinline__ void dgrad_tap_rs(int t, int& r, int& s) const {
    dgrad_tap(a, t, r, s);
  }

  __device__ __forceinline__ const float* image(int b) const {
    return rows ? in + static_cast<int64_t>(rows[b]) * a.in_ld
                : in + static_cast<int64_t>(b) * a.H * a.W * a.C;
  }

  // Forward with channel counts a multiple of 4: four consecutive K of the A
  // row are four channels of one input tap, of the B row four consecutive
  // weights; one 16-byte load each.
  __device__ __forceinline__ void fwd_a(int k, const KCursor& kc, float (&ra)[4]) const {
    const int rs = kc.q, c = kc.r, r = rs / 3, hi = ah + r, wi = aw + rs - 3 * r;
    // bitwise: every term evaluated, no branch (the short-circuit form became
    // exec-mask branches that split the K loop into blocks)
    const bool aok = am & (k < kend) & (hi >= 0) & (hi < a.H) & (wi >= 0) & (wi < a.W);
    const f32x4 va =
        *reinterpret_cast<const f32x4*>(aok ? arow + (hi * a.W + wi) * a.C + c : k_conv_zero);
    for (int e = 0; e < 4; ++e) ra[e] = va[e];
  }
  __device__ __forceinline__ void fwd_b(int k, float (&rb)[4]) const {
    const bool bok = bn & (k < kend);
    const f32x4 vb = *reinterpret_cast<const f32x4*>(
        bok ? Wt + static_cast<int64_t>(bn_idx) * 9 * a.C + k : k_conv_zero);
    for (int e = 0; e < 4; ++e) rb[e] = vb[e];
  }
  __device__ __forceinline__ void fwd_vec(int k, const KCursor& kc, float (&ra)[4],
                                          float (&rb)[4]) const {
    fwd_a(k, kc, ra);
    fwd_b(k, rb);
  }
  // Backward-data A with output channels a multiple of 4 (see dgrad_a).
  __device__ __forceinline__ void dgrad_a_vec(int k, const KCursor& kc, float (&ra)[4]) const {
    const int t = kc.q, o = kc.r;
    int r, sc;
    dgrad_tap_rs(t, r, sc);
    const int ti = ah - r, tj = aw - sc;
    const int i = a.stride == 2 ? ti >> 1 : ti, j = a.stride == 2 ? tj >> 1 : tj;
    const bool ok = am & (k < kend) & (ti >= 0) & (tj >= 0) & (i < a.Ho) & (j < a.Wo);
    const f32x4 v =
        *reinterpret_cast<const f32x4*>(ok ? arow + (i * a.Wo + j) * a.Co + o : k_conv_zero);
    for (int e = 0; e < 4; ++e) ra[e] = v[e];
  }

  // Backward-data operands: A, the output-gradient taps of this input pixel
  // (four consecutive output channels of one tap); B, the weights of this
  // input channel (column) for four consecutive K.
  __device__ __forceinline__ void dgrad_a(int k, float (&ra)[4]) const {
    int t = k / a.Co, o = k - t * a.Co;
    // output-gradient row of tap t for this input pixel, or false where the
    // tap lands outside the output (or, for stride 2 and all nine taps,
    // between output rows)
    auto tap = [&](int t_, int& off) -> bool {
      int r, sc;
      dgrad_tap_rs(t_, r, sc);
      const int ti = ah - r, tj = aw - sc;
      if (ti < 0 || tj < 0) return false;
      int i = ti, j = tj;
      if (a.stride == 2) {
        i = ti >> 1;  // even by the class's choice of taps
        j = tj >> 1;
      }
      if (i >= a.Ho || j >= a.Wo) return false;
      off = (i * a.Wo + j) * a.Co;
      return true;
    };
    if ((a.Co & 3) == 0) {
      f32x4 v = {0.0f, 0.0f, 0.0f, 0.0f};
      int off = 0;
      if (am && k < kend && tap(t, off)) v = *reinterpret_cast<const f32x4*>(arow + off + o);
      for (int e = 0; e < 4; ++e) ra[e] = v[e];
    } else {
      int t2 = t, o2 = o;
      for (int e = 0; e < 4; ++e) {
        int off = 0;
        ra[e] = (am && k + e < kend && tap(t2, off)) ? arow[off + o2] : 0.0f;
        if (++o2 == a.Co) {
          o2 = 0;
          ++t2;
        }
      }
    }
  }
  __device__ __forceinline__ void dgrad_b(int k, float (&rb)[4]) const {
    int t = k / a.Co, o = k - t * a.Co;
    const int K9 = 9 * a.C;
    for (int e = 0; e < 4; ++e) {
      float v = 0.0f;
      if (bn && k + e < kend) {
        int r, sc;
        dgrad_tap_rs(t, r, sc);
        v = Wt[static_cast<int64_t>(o) * K9 + (3 * r + sc) * a.C + bn_idx];
      }
      rb[e] = v;
      if (++o == a.Co) {
        o = 0;
        ++t;
      }
    }
  }

  __device__ __forceinline__ void fetch(int k, float (&ra)[4], float (&rb)[4]) const {
    if constexpr (PASS == CONV_FWD) {
      int rs = k / a.C, c = k - rs * a.C;
      if ((a.C & 3) == 0) {
        f32x4 v = {0.0f, 0.0f, 0.0f, 0.0f};
        const int r = rs / 3, hi = ah + r, wi = aw + rs - 3 * r;
        if (am && k < kend && hi >= 0 && hi < a.H && wi >= 0 && wi < a.W)
          v = *reinterpret_cast<const f32x4*>(arow + (hi * a.W + wi) * a.C + c);
        for (int e = 0; e < 4; ++e) ra[e] = v[e];
      } else {
        for (int e = 0; e < 4; ++e) {
          float v = 0.0f;
          const int r = rs / 3, hi = ah + r, wi = aw + rs - 3 * r;
          if (am && k + e < kend && hi >= 0 && hi < a.H && wi >= 0 && wi < a.W)
            v = arow[(hi * a.W + wi) * a.C + c];
          ra[e] = v;
          if (++c == a.C) {
            c = 0;
            ++rs;
          }
        }
      }
      const int K9 = 9 * a.C;
      if ((K9 & 3) == 0) {
        f32x4 v = {0.0f, 0.0f, 0.0f, 0.0f};
        if (bn && k < kend) v = *reinterpret_cast<const f32x4*>(Wt + static_cast<int64_t>(bn_idx) * K9 + k);
        for (int e = 0; e < 4; ++e) rb[e] = v[e];
      } else {
        for (int e = 0; e < 4; ++e)
          rb[e] = (bn && k + e < kend) ? Wt[static_cast<int64_t>(bn_idx) * K9 + k + e] : 0.0f;
      }
    } else if constexpr (PASS == CONV_DGRAD) {
      dgrad_a(k, ra);
      dgrad_b(k, rb);
    } else if constexpr (PASS == CONV_WGRAD) {
      for (int e = 0; e < 4; ++e)
        ra[e] = (am && k + e < kend) ? dz[static_cast<int64_t>(k + e) * a.Co + am_idx] : 0.0f;
      const int hw = a.Ho * a.Wo;
      int b = k / hw, p = k - b * hw, i = p / a.Wo, j = p - i * a.Wo;
      for (int e = 0; e < 4; ++e) {
        float v = 0.0f;
        if (bn && k + e < kend) {
          if (bones) {
            v = 1.0f;
          } else {
            const int hi = a.stride * i + br - 1, wi = a.stride * j + bs - 1;
            if (hi >= 0 && hi < a.H && wi >= 0 && wi < a.W) v = image(b)[(hi * a.W + wi) * a.C + bc];
          }
        }
        rb[e] = v;
        if (++j == a.Wo) {
          j = 0;
          if (++i == a.Ho) {
            i = 0;
            ++b;
          }
        }
      }
    } else if constexpr (PASS == FC_FWD) {
      for (int e = 0; e < 4; ++e) {
        const bool ok = k + e < kend;
        ra[e] = (am && ok) ? in[am_idx * a.C + k + e] : 0.0f;
        rb[e] = (bn && ok) ? Wt[bn_idx * a.C + k + e] : 0.0f;
      }
    } else if constexpr (PASS == FC_DGRAD) {
      for (int e = 0; e < 4; ++e) {
        const bool ok = k + e < kend;
        ra[e] = (am && ok) ? dz[static_cast<int64_t>(am_idx) * a.dout_ld + k + e] : 0.0f;
        rb[e] = (bn && ok) ? Wt[(k + e) * a.C + bn_idx] : 0.0f;
      }
    } else {  // FC_WGRAD
      for (int e = 0; e < 4; ++e) {
        const bool ok = k + e < kend;
        ra[e] = (am && ok) ? dz[static_cast<int64_t>(k + e) * a.dout_ld + am_idx] : 0.0f;
        rb[e] = (bn && ok) ? (bn_idx == a.C ? 1.0f : in[(k + e) * a.C + bn_idx]) : 0.0f;
      }
    }
  }
};

// Backward-data weights gathered along N (input channels a multiple of 4): a
// thread takes four consecutive input channels nq .. nq + 3 of one K element
// (tap t, output channel o), W[o][r][s][nq .. nq + 3], one 16-byte load.
struct DgradWeightLoader {
  const ConvArgs& a;
  int kend;
  int nq;
  bool bn;
  const float* Wt;
  __device__ DgradWeightLoader(const ConvArgs& a_, int kend_, int n, int N, const float* Wt_)
      : a(a_), kend(kend_), nq(n), bn(n < N), Wt(Wt_) {}
  __device__ __forceinline__ void fetch(int k, const KCursor& kc, float (&rb)[4]) const {
    const int t = kc.q, o = kc.r;
    int r, sc;
    dgrad_tap(a, t, r, sc);
    const bool ok = bn & (k < kend);
    const f32x4 v = *reinterpret_cast<const f32x4*>(
        ok ? Wt + static_cast<int64_t>(o) * 9 * a.C + (3 * r + sc) * a.C + nq : k_conv_zero);
    for (int e = 0; e < 4; ++e) rb[e] = v[e];
  }
};

// Backward-weight loader for channel counts that are multiples of 4.  Both
// operands are contiguous along M or N (dZ is [pixel][Cout], an input tap
// [pixel][Cin]), so a thread gathers, per K step, four consecutive rows of A
// (output channels) and four consecutive columns of B (the channels of one
// tap) of one K element, an output pixel whose position is decoded once for
// both: one 16-byte load each.  With Cin a multiple of 4 a column group lies
// inside one tap, or is the bias column's group (column 9 Cin: ones) or past
// the end.
template <bool GATHER>
struct WgradLoader {
  const ConvArgs& a;
  int kend;
  int mq, nq;         // the thread's first row and column
  bool arow_ok;       // rows mq .. mq + 3 inside (Cout a multiple of 4)
  bool btap, bbias;   // columns: four channels of one tap / the bias group
  int br = 0, bs = 0, bc = 0;  // tap and channel of column nq
  const float* in;
  const int32_t* rows;
  const float* dz;

  __device__ WgradLoader(const ConvArgs& a_, int kend_, int m, int M, int n, int N,
                         const float* in_, const int32_t* rows_, const float* dz_, const float*)
      : a(a_), kend(kend_), mq(m), nq(n), in(in_), rows(rows_), dz(dz_) {
    const int K9 = 9 * a.C;
    arow_ok = mq < M;
    btap = nq < K9;
    bbias = nq == K9 && nq < N;
    const int rs = nq / a.C;
    bc = nq - rs * a.C;
    br = rs / 3;
    bs = rs - 3 * br;
  }

  __device__ __forceinline__ void fetch(int k, const PixCursor& pc, float (&ra)[4],
                                        float (&rb)[4]) const {
    const bool ok = k < kend;
    const int b = ok ? pc.b : 0, i = pc.i, j = pc.j;  // a valid image past the end
    const f32x4 va = *reinterpret_cast<const f32x4*>(
        ok && arow_ok ? dz + static_cast<int64_t>(k) * a.Co + mq : k_conv_zero);
    const int hi = a.stride * i + br - 1, wi = a.stride * j + bs - 1;
    const bool tap_ok = ok & btap & (hi >= 0) & (hi < a.H) & (wi >= 0) & (wi < a.W);
    // the gathered case is a template parameter: a branch on `rows` here made
    // the compiler wait for every load in flight (the next steps' too) before
    // each LDS store
    const float* img;
    if constexpr (GATHER)
      img = in + static_cast<int64_t>(rows[b]) * a.in_ld;
    else
      img = in + static_cast<int64_t>(b) * a.H * a.W * a.C;
    const f32x4 vb = *reinterpret_cast<const f32x4*>(
        tap_ok ? img + (hi * a.W + wi) * a.C + bc : k_conv_zero);
    for (int e = 0; e < 4; ++e) {
      ra[e] = va[e];
      rb[e] = vb[e];
    }
    rb[0] = ok && bbias ? 1.0f : rb[0];
  }
};

// Channel counts for the vector loaders (conv_gemm_kernel<PASS, true>).
__host__ __device__ inline bool vector_loaders(const ConvArgs& a) {
  return (a.C & 3) == 0 && (a.Co & 3) == 0;
}

// Tiles of one stride-2 backward-data class.
__host__ __device__ inline int64_t dgrad_class_tiles(ConvArgs a, int cls) {
  a.cls = cls;
  const Dims d = pass_dims(a, CONV_DGRAD);
  return ((d.M + CT - 1) / CT) * ((d.N + CT - 1) / CT);
}
// The classes of a stride-2 backward-data launch in workgroup order: the
// most taps (longest K) first, so that the short ones fill the last pass.
__host__ __device__ inline int dgrad_class_at(int i) { return i == 0 ? 3 : i == 1 ? 1 : i == 2 ? 2 : 0; }

// TR (channel counts multiples of 4, see vector_loaders): vector loaders
// without branches around their loads -- the forward gathers along K as
// ConvLoader does, backward-weight gathers both operands along M and N
// (WgradLoader), backward-data its weights along N (DgradWeightLoader);
// otherwise ConvLoader's general gathers along K.
// One tile of the GEMM; `lds` holds 4 HALVES CK CLD floats (conv_gemm_kernel,
// conv_bwd_pair_kernel).
template <int PASS, bool TR, int HALVES, bool GATHER>
__device__ __forceinline__ void conv_gemm_tile(ConvArgs a, int tile, float* lds) {
  constexpr bool WG = PASS == CONV_WGRAD || PASS == FC_WGRAD;
  static_assert(HALVES == 1 || HALVES == 2, "K per step: CK or 2 CK");
  constexpr int KS = HALVES * CK;  // K per step (one barrier)
  typedef float Stage[2][KS][CLD];
  Stage& As = *reinterpret_cast<Stage*>(lds);
  Stage& Bs = *reinterpret_cast<Stage*>(lds + 2 * KS * CLD);
  int split = 0;
  if constexpr (PASS == CONV_DGRAD) {
    if (a.stride == 2 && a.cls < 0) {
      // all four parity classes in one launch: the workgroup's class and its
      // tile within the class
      int i = 0;
      for (; i < 4; ++i) {
        const int t = static_cast<int>(dgrad_class_tiles(a, dgrad_class_at(i)));
        if (tile < t) break;
        tile -= t;
      }
      if (i == 4) return;  // past the last class (the grid is their sum)
      a.cls = dgrad_class_at(i);
    }
  }
  const Dims d = pass_dims(a, PASS);
  const int M = static_cast<int>(d.M), N = static_cast<int>(d.N), K = static_cast<int>(d.K);
  const int z = blockIdx.y;
  const int rep = a.order[z];
  const int gm = (M + CT - 1) / CT, gn = (N + CT - 1) / CT;
  if constexpr (WG) {
    split = tile / (gm * gn);
    tile -= split * gm * gn;
  }
  const int m0 = tile / gn * CT, n0 = (tile - tile / gn * gn) * CT;
  const int kbeg = WG ? split * static_cast<int>(a.k_per_split) : 0;
  const int kend = WG ? (K - kbeg < a.k_per_split ? K : kbeg + static_cast<int>(a.k_per_split)) : K;

  const float* in = a.in ? a.in + z * a.in_slot : nullptr;
  const int32_t* rows = a.gather ? a.gather + z * a.gather_slot : nullptr;
  const float* dz = a.dout ? a.dout + z * a.dout_slot : nullptr;
  const float* par = a.master_in + static_cast<int64_t>(rep) * a.master_in_slot;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, r = lane & 31, h = lane >> 5;
  // a thread's share of each K step: one row of A and of B and four
  // consecutive K (lr, lk .. lk + 3), or, for backward-weight, four
  // consecutive rows and columns (lr .. lr + 3) and one K (lk)
  static_assert(!TR || PASS == CONV_FWD || PASS == CONV_WGRAD || PASS == CONV_DGRAD,
                "vector loaders: convolution passes");
  constexpr bool TRA = TR && PASS == CONV_WGRAD;  // A gathered along M
  constexpr bool TRB = TR && PASS != CONV_FWD;    // B gathered along N
  // (lr, lk): the thread's A row and K offset, (lrb, lkb) its B row and K
  // offset; four consecutive K of one row, or four consecutive rows of one K
  const int lr = TRA ? 4 * (tid & 15) : tid >> 2;
  const int lk = TRA ? tid >> 4 : (tid & 3) * 4;
  const int lrb = TRB ? 4 * (tid & 15) : tid >> 2;
  const int lkb = TRB ? tid >> 4 : (tid & 3) * 4;
  typedef typename std::conditional<TRA, WgradLoader<GATHER>, ConvLoader<PASS>>::type Loader;
  const Loader ld(a, kend, m0 + lr, M, n0 + lrb, N, in, rows, dz, par + a.w_off);
  const DgradWeightLoader wl(a, kend, n0 + lrb, N, par + a.w_off);
  // the vector loaders' K decode, stepped along with the loads (consecutive K
  // steps; one cursor per half of a step)
  const int kdiv = PASS == CONV_FWD ? a.C : a.Co;
  const int ho = a.Ho > 0 ? a.Ho : 1, wo = a.Wo > 0 ? a.Wo : 1;
  KCursor ka[HALVES] = {KCursor(kbeg + lk, kdiv, KS)};
  KCursor kb[HALVES] = {KCursor(kbeg + lkb, a.Co, KS)};
  PixCursor pc[HALVES] = {PixCursor(TRA ? kbeg + lk : 0, ho, wo, KS)};
  if constexpr (HALVES == 2) {
    ka[1] = KCursor(kbeg + CK + lk, kdiv, KS);
    kb[1] = KCursor(kbeg + CK + lkb, a.Co, KS);
    pc[1] = PixCursor(TRA ? kbeg + CK + lk : 0, ho, wo, KS);
  }
  float ra[2][HALVES][4], rb[2][HALVES][4];
  auto load = [&](int k0, auto P) {
    constexpr int p = decltype(P)::value;
#pragma unroll
    for (int q = 0; q < HALVES; ++q) {
      const int kq = k0 + q * CK;
      if constexpr (TR && PASS == CONV_DGRAD) {
        ld.dgrad_a_vec(kq + lk, ka[q], ra[p][q]);
        wl.fetch(kq + lkb, kb[q], rb[p][q]);
        ka[q].next();
        kb[q].next();
      } else if constexpr (TR && PASS == CONV_FWD) {
        ld.fwd_vec(kq + lk, ka[q], ra[p][q], rb[p][q]);
        ka[q].next();
      } else if constexpr (TRA) {
        ld.fetch(kq + lk, pc[q], ra[p][q], rb[p][q]);
        pc[q].next();
      } else {
        ld.fetch(kq + lk, ra[p][q], rb[p][q]);
      }
    }
  };
  auto stash = [&](auto P) {
    constexpr int p = decltype(P)::value;  // register set p into LDS buffer p
#pragma unroll
    for (int q = 0; q < HALVES; ++q) {
      const int kq = q * CK;
      if constexpr (TRA) {
        *reinterpret_cast<f32x4*>(&As[p][kq + lk][lr]) =
            f32x4{ra[p][q][0], ra[p][q][1], ra[p][q][2], ra[p][q][3]};
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) As[p][kq + lk + e][lr] = ra[p][q][e];
      }
      if constexpr (TRB) {
        *reinterpret_cast<f32x4*>(&Bs[p][kq + lkb][lrb]) =
            f32x4{rb[p][q][0], rb[p][q][1], rb[p][q][2], rb[p][q][3]};
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) Bs[p][kq + lkb + e][lrb] = rb[p][q][e];
      }
    }
  };

  f32x16 acc;
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.0f;
  const int nk = (kend - kbeg + KS - 1) / KS;
  // Two register sets: step t + 2 is gathered while step t is multiplied and
  // step t + 1 (gathered a step earlier) goes into the other LDS buffer.
  // Gathers past kend read nothing and give zeros.
  load(kbeg, Pi<0>());
  stash(Pi<0>());
  load(kbeg + KS, Pi<1>());
  __syncthreads();
  // a wave whose 32 x 32 block lies wholly past M or N (32-channel layers on
  // 64 x 64 tiles) skips its products and leaves the MFMA unit to the CU's
  // other workgroups
  const bool busy = m0 + wm * 32 < M && n0 + wn * 32 < N;
  auto step = [&](int t, auto P, auto MUL) {  // register set and LDS buffer p = t & 1
    constexpr int p = decltype(P)::value;
    load(kbeg + (t + 2) * KS, P);
    // MFMA u contracts k = 2u (lanes 0-31) and 2u + 1 (lanes 32-63)
    if constexpr (decltype(MUL)::value) {
#pragma unroll
      for (int u = 0; u < KS / 2; ++u)
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(As[p][2 * u + h][wm * 32 + r],
                                                   Bs[p][2 * u + h][wn * 32 + r], acc, 0, 0, 0);
    }
    stash(Pi<p ^ 1>());
    if constexpr (decltype(MUL)::value) interleave<KS / 2>();
    __syncthreads();
  };
  auto steps = [&](auto MUL) {
    int t = 0;
    for (; t + 1 < nk; t += 2) {
      step(t, Pi<0>(), MUL);
      step(t + 1, Pi<1>(), MUL);
    }
    if (t < nk) step(t, Pi<0>(), MUL);
  };
  if (busy)
    steps(Pi<1>());
  else
    steps(Pi<0>());  // loads, stores and barriers only

  // accumulator i of lane (r, h): row 8 (i / 4) + 4 h + i % 4, column r
  const int col = n0 + wn * 32 + r;
  if constexpr (PASS == CONV_DGRAD) {
    // the rows' input pixels by stepping: +1 within a group of four, +5 between
    DgradRowWalker wk(a, m0 + wm * 32 + 4 * h);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (i > 0) wk.advance((i & 3) ? 1 : 5);
      const int row = m0 + wm * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
      if (row >= M || col >= N) continue;
      const int64_t at = wk.offset() + col;
      const float g = a.skip ? acc[i] + a.skip[z * a.skip_slot + at] : acc[i];
      a.out[z * a.out_slot + at] = a.mask[z * a.mask_slot + at] > 0.0f ? g : 0.0f;
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int row = m0 + wm * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
    if (row >= M || col >= N) continue;
    const float v = acc[i];
    if constexpr (PASS == CONV_FWD) {
      const int64_t at = static_cast<int64_t>(row) * a.Co + col;
      float zv = v + par[a.b_off + col];
      if (a.skip) zv += a.skip[z * a.skip_slot + at];
      a.out[z * a.out_slot + at] = zv > 0.0f ? zv : 0.0f;
    } else if constexpr (PASS == FC_FWD) {
      a.out[z * a.out_slot + static_cast<int64_t>(row) * a.out_ld + col] = v + par[a.b_off + col];
    } else if constexpr (PASS == FC_DGRAD) {
      a.out[z * a.out_slot + static_cast<int64_t>(row) * a.out_ld + col] = v;
    } else {
      a.part[z * a.part_slot + (static_cast<int64_t>(split) * M + row) * N + col] = v;
    }
  }
}

template <int PASS, bool TR = false, int HALVES = 1, bool GATHER = false>
__global__ __launch_bounds__(256) void conv_gemm_kernel(ConvArgs a) {
  __shared__ __attribute__((aligned(16))) float lds[4 * HALVES * CK * CLD];
  conv_gemm_tile<PASS, TR, HALVES, GATHER>(a, blockIdx.x, lds);
}

// ---------------------------------------------------------------------------
// Backward-data with at most 32 input channels (a multiple of 4): 128 x 32
// tiles, the four waves stacked along M, where a 64 x 64 tile would leave half
// of its columns empty.  The operands are gathered as in
// conv_gemm_kernel<CONV_DGRAD, true> (each thread two A rows, four
// consecutive K of each; the first 128 threads four consecutive weight
// columns of one K), the LDS tiles hold the same K steps, and so every sum
// is the same.
constexpr int NM = 128, NN = 32;

__host__ __device__ inline bool dgrad_narrow(const ConvArgs& a) {
  return (a.C & 3) == 0 && (a.Co & 3) == 0 && a.C >= 4 && a.C <= NN;
}
__host__ __device__ inline int64_t dgrad_narrow_tiles(const ConvArgs& a) {
  const Dims d = pass_dims(a, CONV_DGRAD);
  return ((d.M + NM - 1) / NM) * ((d.N + NN - 1) / NN);
}

// `lds` holds 2 CK (NM + NN + 8) floats.
__device__ __forceinline__ void conv_dgrad_narrow_tile(ConvArgs a, int tile, float* lds) {
  typedef float StageA[2][CK][NM + 4];
  typedef float StageB[2][CK][NN + 4];
  StageA& As = *reinterpret_cast<StageA*>(lds);
  StageB& Bs = *reinterpret_cast<StageB*>(lds + 2 * CK * (NM + 4));
  if (a.stride == 2 && a.cls < 0) {
    int i = 0;
    for (; i < 4; ++i) {
      ConvArgs ac = a;
      ac.cls = dgrad_class_at(i);
      const int t = static_cast<int>(dgrad_narrow_tiles(ac));
      if (tile < t) break;
      tile -= t;
    }
    if (i == 4) return;  // past the last class (the grid is their sum)
    a.cls = dgrad_class_at(i);
  }
  const Dims d = pass_dims(a, CONV_DGRAD);
  const int M = static_cast<int>(d.M), N = static_cast<int>(d.N), K = static_cast<int>(d.K);
  const int z = blockIdx.y;
  const int rep = a.order[z];
  const int gn = (N + NN - 1) / NN;
  const int m0 = tile / gn * NM, n0 = (tile - tile / gn * gn) * NN;
  const float* dz = a.dout + z * a.dout_slot;
  const float* par = a.master_in + static_cast<int64_t>(rep) * a.master_in_slot;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, r = lane & 31, h = lane >> 5;
  const int lr = tid >> 2, lk = (tid & 3) * 4;      // A rows lr and lr + 64
  const bool bload = tid < NN * CK / 4;             // B: four columns of one K
  const int lrb = 4 * (tid & 7), lkb = (tid >> 3) & (CK - 1);
  const ConvLoader<CONV_DGRAD> ld0(a, K, m0 + lr, M, n0, N, nullptr, nullptr, dz, par + a.w_off);
  const ConvLoader<CONV_DGRAD> ld1(a, K, m0 + lr + 64, M, n0, N, nullptr, nullptr, dz,
                                   par + a.w_off);
  const DgradWeightLoader wl(a, K, n0 + lrb, N, par + a.w_off);
  KCursor ka(lk, a.Co), kb(lkb, a.Co);  // stepped along with the loads
  float ra0[4], ra1[4], rb[4];
  auto load = [&](int k0) {
    ld0.dgrad_a_vec(k0 + lk, ka, ra0);
    ld1.dgrad_a_vec(k0 + lk, ka, ra1);
    if (bload) wl.fetch(k0 + lkb, kb, rb);
    ka.next();
    kb.next();
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      As[buf][lk + e][lr] = ra0[e];
      As[buf][lk + e][lr + 64] = ra1[e];
    }
    if (bload) *reinterpret_cast<f32x4*>(&Bs[buf][lkb][lrb]) = f32x4{rb[0], rb[1], rb[2], rb[3]};
  };

  f32x16 acc;
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.0f;
  const int nk = (K + CK - 1) / CK;
  load(0);
  stash(0);
  __syncthreads();
  for (int t = 0; t < nk; ++t) {
    const int buf = t & 1;
    if (t + 1 < nk) load((t + 1) * CK);
#pragma unroll
    for (int u = 0; u < CK / 2; ++u)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(As[buf][2 * u + h][wave * 32 + r],
                                                 Bs[buf][2 * u + h][r], acc, 0, 0, 0);
    if (t + 1 < nk) stash(buf ^ 1);
    interleave<CK / 2>();
    __syncthreads();
  }

  const int col = n0 + r;
  DgradRowWalker wk(a, m0 + wave * 32 + 4 * h);  // stepped as in conv_gemm_kernel
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    if (i > 0) wk.advance((i & 3) ? 1 : 5);
    const int row = m0 + wave * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
    if (row >= M || col >= N) continue;
    const int64_t at = wk.offset() + col;
    const float g = a.skip ? acc[i] + a.skip[z * a.skip_slot + at] : acc[i];
    a.out[z * a.out_slot + at] = a.mask[z * a.mask_slot + at] > 0.0f ? g : 0.0f;
  }
}

__global__ __launch_bounds__(256) void conv_dgrad_narrow_kernel(ConvArgs a) {
  __shared__ __attribute__((aligned(16))) float lds[2 * CK * (NM + NN + 8)];
  conv_dgrad_narrow_tile(a, blockIdx.x, lds);
}

// ---------------------------------------------------------------------------
// Forward into at most 32 output channels and backward-weight of at most 32
// output channels (channel counts multiples of 4, at least 4 input channels),
// where a 64 x 64 tile would leave half of its waves without products:
//   forward          128 x 32 tiles (pixels x output channels), the four waves
//                    stacked along M; each thread gathers two A rows and, in
//                    the first 128 threads, one weight row, four consecutive K
//                    each, as conv_gemm_kernel<CONV_FWD, true> does;
//   backward-weight  32 x 128 tiles (output channels x weight columns), the
//                    waves side by side along N; each thread takes one K (an
//                    output pixel) and, as WgradLoader does, four output
//                    channels (the first eight threads of each K) and two
//                    groups of four weight columns.
// Both keep the LDS layout of the 64 x 64 tiles (K steps of CK, [k][row]) and
// the operand roles of every MFMA, and so every sum is the same.  Two
// register sets as there: step t + 2 is gathered while step t is multiplied.
__host__ __device__ inline bool conv_narrow(const ConvArgs& a) {
  return (a.C & 3) == 0 && (a.Co & 3) == 0 && a.C >= 4 && a.Co <= NN;
}
__host__ __device__ inline int64_t fwd_narrow_tiles(const ConvArgs& a) {
  const Dims d = pass_dims(a, CONV_FWD);
  return ((d.M + NM - 1) / NM) * ((d.N + NN - 1) / NN);
}
__host__ __device__ inline int64_t wgrad_narrow_tiles(const ConvArgs& a) {
  const Dims d = pass_dims(a, CONV_WGRAD);
  return ((d.M + NN - 1) / NN) * ((d.N + NM - 1) / NM);
}

__global__ __launch_bounds__(256) void conv_fwd_narrow_kernel(ConvArgs a) {
  __shared__ __attribute__((aligned(16))) float As[2][CK][NM + 4];
  __shared__ __attribute__((aligned(16))) float Bs[2][CK][NN + 4];
  const Dims d = pass_dims(a, CONV_FWD);
  const int M = static_cast<int>(d.M), N = static_cast<int>(d.N), K = static_cast<int>(d.K);
  const int z = blockIdx.y;
  const int rep = a.order[z];
  const int gn = (N + NN - 1) / NN;
  const int tile = blockIdx.x;
  const int m0 = tile / gn * NM, n0 = (tile - tile / gn * gn) * NN;
  const float* in = a.in + z * a.in_slot;
  const int32_t* rows = a.gather ? a.gather + z * a.gather_slot : nullptr;
  const float* par = a.master_in + static_cast<int64_t>(rep) * a.master_in_slot;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, r = lane & 31, h = lane >> 5;
  // A rows lr and lr + 64, B row lr (threads below 128), K lk .. lk + 3
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  const bool bload = tid < NN * CK / 4;
  const ConvLoader<CONV_FWD> ld0(a, K, m0 + lr, M, n0 + lr, N, in, rows, nullptr, par + a.w_off);
  const ConvLoader<CONV_FWD> ld1(a, K, m0 + lr + 64, M, n0 + lr, N, in, rows, nullptr,
                                 par + a.w_off);
  KCursor ka(lk, a.C);  // stepped along with the loads
  float ra0[2][4], ra1[2][4], rb[2][4];
  auto load = [&](int k0, auto P) {
    constexpr int p = decltype(P)::value;
    ld0.fwd_a(k0 + lk, ka, ra0[p]);
    ld1.fwd_a(k0 + lk, ka, ra1[p]);
    ld0.fwd_b(k0 + lk, rb[p]);  // rows past N (threads from 128 on) read zeros
    ka.next();
  };
  auto stash = [&](auto P) {
    constexpr int p = decltype(P)::value;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      As[p][lk + e][lr] = ra0[p][e];
      As[p][lk + e][lr + 64] = ra1[p][e];
    }
    if (bload) {
#pragma unroll
      for (int e = 0; e < 4; ++e) Bs[p][lk + e][lr] = rb[p][e];
    }
  };

  f32x16 acc;
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.0f;
  const int nk = (K + CK - 1) / CK;
  load(0, Pi<0>());
  stash(Pi<0>());
  load(CK, Pi<1>());
  __syncthreads();
  auto step = [&](int t, auto P) {
    constexpr int p = decltype(P)::value;
    load((t + 2) * CK, P);
#pragma unroll
    for (int u = 0; u < CK / 2; ++u)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(As[p][2 * u + h][wave * 32 + r],
                                                 Bs[p][2 * u + h][r], acc, 0, 0, 0);
    stash(Pi<p ^ 1>());
    interleave<CK / 2>();
    __syncthreads();
  };
  int t = 0;
  for (; t + 1 < nk; t += 2) {
    step(t, Pi<0>());
    step(t + 1, Pi<1>());
  }
  if (t < nk) step(t, Pi<0>());

  const int col = n0 + r;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int row = m0 + wave * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
    if (row >= M || col >= N) continue;
    const int64_t at = static_cast<int64_t>(row) * a.Co + col;
    float zv = acc[i] + par[a.b_off + col];
    if (a.skip) zv += a.skip[z * a.skip_slot + at];
    a.out[z * a.out_slot + at] = zv > 0.0f ? zv : 0.0f;
  }
}

// `lds` holds 2 CK (NM + NN + 8) floats.
template <bool GATHER>
__device__ __forceinline__ void conv_wgrad_narrow_tile(ConvArgs a, int tile, float* lds) {
  typedef float StageA[2][CK][NN + 4];
  typedef float StageB[2][CK][NM + 4];
  StageA& As = *reinterpret_cast<StageA*>(lds);
  StageB& Bs = *reinterpret_cast<StageB*>(lds + 2 * CK * (NN + 4));
  const Dims d = pass_dims(a, CONV_WGRAD);
  const int M = static_cast<int>(d.M), N = static_cast<int>(d.N), K = static_cast<int>(d.K);
  const int z = blockIdx.y;
  const int rep = a.order[z];
  const int gm = (M + NN - 1) / NN, gn = (N + NM - 1) / NM;
  const int split = tile / (gm * gn);
  tile -= split * gm * gn;
  const int m0 = tile / gn * NN, n0 = (tile - tile / gn * gn) * NM;
  const int kbeg = split * static_cast<int>(a.k_per_split);
  const int kend = K - kbeg < a.k_per_split ? K : kbeg + static_cast<int>(a.k_per_split);
  const float* in = a.in + z * a.in_slot;
  const int32_t* rows = a.gather ? a.gather + z * a.gather_slot : nullptr;
  const float* dz = a.dout + z * a.dout_slot;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, r = lane & 31, h = lane >> 5;
  // K lk; A rows 4 q .. 4 q + 3 (q below 8); B columns 4 q .. + 3 and 64 + 4 q .. + 3
  const int lk = tid >> 4, q = tid & 15;
  const bool aload = q < NN / 4;
  const WgradLoader<GATHER> w0(a, kend, aload ? m0 + 4 * q : M, M, n0 + 4 * q, N, in, rows, dz,
                              nullptr);
  const WgradLoader<GATHER> w1(a, kend, M, M, n0 + 64 + 4 * q, N, in, rows, dz, nullptr);
  PixCursor pc(kbeg + lk, a.Ho, a.Wo);
  float ra[2][4], rb0[2][4], rb1[2][4];
  auto load = [&](int k0, auto P) {
    constexpr int p = decltype(P)::value;
    float unused[4];
    w0.fetch(k0 + lk, pc, ra[p], rb0[p]);
    w1.fetch(k0 + lk, pc, unused, rb1[p]);  // its A rows are past M: zeros, not stored
    pc.next();
  };
  auto stash = [&](auto P) {
    constexpr int p = decltype(P)::value;
    if (aload)
      *reinterpret_cast<f32x4*>(&As[p][lk][4 * q]) = f32x4{ra[p][0], ra[p][1], ra[p][2], ra[p][3]};
    *reinterpret_cast<f32x4*>(&Bs[p][lk][4 * q]) =
        f32x4{rb0[p][0], rb0[p][1], rb0[p][2], rb0[p][3]};
    *reinterpret_cast<f32x4*>(&Bs[p][lk][64 + 4 * q]) =
        f32x4{rb1[p][0], rb1[p][1], rb1[p][2], rb1[p][3]};
  };

  f32x16 acc;
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.0f;
  const int nk = (kend - kbeg + CK - 1) / CK;
  load(kbeg, Pi<0>());
  stash(Pi<0>());
  load(kbeg + CK, Pi<1>());
  __syncthreads();
  // a wave whose 32 columns lie past N (the last tile) skips its products
  const bool busy = n0 + wave * 32 < N;
  auto step = [&](int t, auto P, auto MUL) {
    constexpr int p = decltype(P)::value;
    load(kbeg + (t + 2) * CK, P);
    if constexpr (decltype(MUL)::value) {
#pragma unroll
      for (int u = 0; u < CK / 2; ++u)
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(As[p][2 * u + h][r],
                                                   Bs[p][2 * u + h][wave * 32 + r], acc, 0, 0, 0);
    }
    stash(Pi<p ^ 1>());
    if constexpr (decltype(MUL)::value) interleave<CK / 2>();
    __syncthreads();
  };
  auto steps = [&](auto MUL) {
    int t = 0;
    for (; t + 1 < nk; t += 2) {
      step(t, Pi<0>(), MUL);
      step(t + 1, Pi<1>(), MUL);
    }
    if (t < nk) step(t, Pi<0>(), MUL);
  };
  if (busy)
    steps(Pi<1>());
  else
    steps(Pi<0>());

  const int col = n0 + wave * 32 + r;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int row = m0 + 8 * (i >> 2) + 4 * h + (i & 3);
    if (row >= M || col >= N) continue;
    a.part[z * a.part_slot + (static_cast<int64_t>(split) * M + row) * N + col] = acc[i];
  }
}

template <bool GATHER>
__global__ __launch_bounds__(256) void conv_wgrad_narrow_kernel(ConvArgs a) {
  __shared__ __attribute__((aligned(16))) float lds[2 * CK * (NM + NN + 8)];
  conv_wgrad_narrow_tile<GATHER>(a, blockIdx.x, lds);
}

// Backward-data and backward-weight of one layer in one launch: the first nd
// workgroups take backward-data tiles, the others backward-weight tiles.  The
// two read the layer's output gradient and nothing that the other writes;
// with one or two replicas either launch alone leaves most of every CU idle,
// and with more the two kinds of tiles share the CUs better than in turn.
// DN / WN: the 128 x 32 backward-data / 32 x 128 backward-weight tiles, else
// the 64 x 64 ones (vector loaders, K steps of CK).
template <bool DN, bool WN>
__global__ __launch_bounds__(256) void conv_bwd_pair_kernel(ConvArgs d, ConvArgs w, int nd) {
  constexpr int DF = DN ? 2 * CK * (NM + NN + 8) : 4 * CK * CLD;
  constexpr int WF = WN ? 2 * CK * (NM + NN + 8) : 4 * CK * CLD;
  __shared__ __attribute__((aligned(16))) float lds[DF > WF ? DF : WF];
  const int b = blockIdx.x;
  if (b < nd) {
    if constexpr (DN)
      conv_dgrad_narrow_tile(d, b, lds);
    else
      conv_gemm_tile<CONV_DGRAD, true, 1, false>(d, b, lds);
  } else {
    if constexpr (WN)
      conv_wgrad_narrow_tile<false>(w, b - nd, lds);
    else
      conv_gemm_tile<CONV_WGRAD, true, 1, false>(w, b - nd, lds);
  }
}

// ---------------------------------------------------------------------------
// Thin input layers (at most 3 input channels, at most 32 output channels in
// fours; layer 1 of an RGB network).  Their GEMMs are too narrow for 64 x 64
// tiles (K = 9 Cin <= 27 in the forward, N = 9 Cin + 1 in backward-weight) and
// their input channels too few for vector gathers, so they get kernels of
// their own.  (Backward-data is never needed: layer 1 has no layer below.)

__host__ __device__ inline bool thin_layer(const ConvArgs& a) {
  return a.C >= 1 && a.C <= 3 && a.Co >= 4 && a.Co <= 32 && (a.Co & 3) == 0;
}

// Forward on the fp32 MFMA: Z[p][o] = (sum over the taps t = (3 r + s) Cin + c
// of in(tap) W[o][t]) + b[o], then ReLU.  A 32 x 32 block is 32 output pixels
// (rows) by the output channels (columns; zero weights past Cout).  K is the
// 9 Cin taps padded to 2 J: MFMA j contracts tap j (lanes 0-31) and tap J + j
// (lanes 32-63).  Each lane keeps its column's J weights in registers and
// gathers its pixel's taps straight from memory; a wave takes TB consecutive
// blocks and loads all their taps before its first MFMA.  A store of one
// accumulator register writes two output pixels' channels (whole lines).
constexpr int THIN_TB = 2;
constexpr int tap_rs(int t, int cin) { return t / cin; }
constexpr int tap_c(int t, int cin) { return t % cin; }

template <int CIN>
__global__ __launch_bounds__(256) void conv_thin_fwd_kernel(ConvArgs a) {
  constexpr int KT = 9 * CIN, J = (KT + 1) / 2;
  const int z = blockIdx.y;
  const int lane = threadIdx.x & 63, l32 = lane & 31, h = lane >> 5;
  const float* par = a.master_in + static_cast<int64_t>(a.order[z]) * a.master_in_slot;
  const bool col_ok = l32 < a.Co;
  float wv[J];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int t = j + J * h;
    wv[j] = *(col_ok && t < KT ? par + a.w_off + static_cast<int64_t>(l32) * KT + t
                               : k_conv_zero);
  }
  const float bias = *(col_ok ? par + a.b_off + l32 : k_conv_zero);
  const int hw = a.Ho * a.Wo;
  const int64_t M = static_cast<int64_t>(a.B) * hw;
  const int64_t p0 =
      (static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6)) * (32 * THIN_TB);
  const float* in = a.in + z * a.in_slot;
  float xv[THIN_TB][J];
#pragma unroll
  for (int u = 0; u < THIN_TB; ++u) {
    const int64_t p = p0 + 32 * u + l32;
    const bool pok = p < M;
    const int64_t ps = pok ? p : 0;
    const int b = static_cast<int>(ps / hw);
    const int q = static_cast<int>(ps - static_cast<int64_t>(b) * hw);
    const int i = q / a.Wo, jj = q - i * a.Wo;
    const float* img =
        a.gather ? in + static_cast<int64_t>(a.gather[z * a.gather_slot + b]) * a.in_ld
                 : in + static_cast<int64_t>(b) * a.H * a.W * CIN;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      // tap j or J + j: (r, s) and channel fixed at compile time for each half
      const int rs = h ? tap_rs(j + J, CIN) : tap_rs(j, CIN);
      const int c = h ? tap_c(j + J, CIN) : tap_c(j, CIN);
      const int r = rs / 3, sc = rs - 3 * r;
      const int hi = a.stride * i + r - 1, wi = a.stride * jj + sc - 1;
      const bool ok = pok && j + J * h < KT && hi >= 0 && hi < a.H && wi >= 0 && wi < a.W;
      xv[u][j] = *(ok ? img + (hi * a.W + wi) * CIN + c : k_conv_zero);
    }
  }
  float* out = a.out + z * a.out_slot;
#pragma unroll
  for (int u = 0; u < THIN_TB; ++u) {
    f32x16 acc;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
#pragma unroll
    for (int j = 0; j < J; ++j) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(xv[u][j], wv[j], acc, 0, 0, 0);
    // accumulator e of lane (l32, h): pixel row 8 (e / 4) + 4 h + e % 4, channel l32
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int64_t p = p0 + 32 * u + 8 * (e >> 2) + 4 * h + (e & 3);
      const float v = acc[e] + bias;
      if (p < M && col_ok) out[p * a.Co + l32] = v > 0.0f ? v : 0.0f;
    }
  }
}

// Backward-weight partial of one range of whole output rows (workgroup =
// range): C[o][n] = sum over the range's pixels p of dZ[p][o] x(p, n), with
// x(p, n) the input tap of column n < 9 Cin and 1 for the bias column.  The
// input rows the range's taps read are staged in LDS first, zero-padded:
// for range row q and tap row r, input row stride i + r - 1 of its image,
// with a zero column on the left and zeros past the right edge up to the
// last column a 32-pixel block of the row can reach.  A tap then needs no
// bounds test and its LDS offset steps by a constant from pixel to pixel.
// The whole 32 x 32 block is one MFMA accumulator: wave w takes range rows
// w, w + 4, ..., each in blocks of 32 pixels, one 32x32x2 fp32 MFMA per
// pixel pair (lane l holds dZ[p + l / 32][l % 32] and x(p + l / 32, l % 32)),
// dZ of the next block loaded while the current one is multiplied; the four
// waves' sums are added in wave order.
constexpr int THIN_WG_PIXELS = 512;   // a range's pixel slots (rows x padded width) at most
// The forward's workgroups take the same ranges (ranges of 128 or 256 pixel
// slots, more workgroups, ran the first layer of a 32 x 32 x 3 network slower over a round).
constexpr int THIN_FWD_PIXELS = THIN_WG_PIXELS;
constexpr int THIN_STAGE_MAX = 11264;  // staged floats at most (44 KB, with red: under 64 KB)

__host__ __device__ inline int thin_wo_pad(const ConvArgs& a) { return (a.Wo + 31) / 32 * 32; }
__host__ __device__ inline int thin_rows_per_range(const ConvArgs& a, int pixels = THIN_WG_PIXELS) {
  const int r = pixels / thin_wo_pad(a);
  return r > 1 ? r : 1;
}
__host__ __device__ inline int thin_row_width(const ConvArgs& a) {
  return a.stride * thin_wo_pad(a) + 2;
}
__host__ __device__ inline int64_t thin_stage_floats(const ConvArgs& a, int pixels = THIN_WG_PIXELS) {
  return static_cast<int64_t>(thin_rows_per_range(a, pixels)) * 3 * thin_row_width(a) * a.C;
}
__host__ __device__ inline bool thin_wgrad(const ConvArgs& a) {
  return thin_layer(a) && (a.stride == 1 || a.stride == 2) && thin_stage_floats(a) <= THIN_STAGE_MAX;
}

// Stages the input rows of range rows [r0, r0 + nr_rows) in LDS, zero-padded
// (x_s[(3 q + r) per_row + col CIN + c] = input row STRIDE i + r - 1, column
// col - 1, of range row q's image, or 0): first the source offset of every
// staged row (-1: a padding row), then the elements, eight loads per thread
// in flight (a padding element reads the zero array).  Ends with a barrier.
template <int CIN, int STRIDE>
__device__ __forceinline__ void thin_stage(const ConvArgs& a, int z, int r0, int R, int nr_rows,
                                           int per_row, float* x_s) {
  __shared__ int64_t src_s[3 * (THIN_WG_PIXELS / 32)];
  const float* in = a.in + z * a.in_slot;
  if (threadIdx.x < 3 * R) {
    const int sr = threadIdx.x, q = sr / 3, r = sr - 3 * q;
    int64_t off = -1;
    if (q < nr_rows) {
      const int orow = r0 + q, b = orow / a.Ho, i = orow - b * a.Ho;
      const int hi = STRIDE * i + r - 1;
      if (hi >= 0 && hi < a.H) {
        const int64_t img = a.gather ? static_cast<int64_t>(a.gather[z * a.gather_slot + b]) * a.in_ld
                                     : static_cast<int64_t>(b) * a.H * a.W * CIN;
        off = img + static_cast<int64_t>(hi) * a.W * CIN;
      }
    }
    src_s[sr] = off;
  }
  __syncthreads();
  const int n_stage = 3 * R * per_row;
  KCursor ec(threadIdx.x, per_row, 256);  // element e = staged row q, column r
  for (int e0 = threadIdx.x; e0 < n_stage; e0 += 8 * 256) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = e0 + 256 * u;
      const int col = ec.r;
      const int64_t off = src_s[e < n_stage ? ec.q : 0];
      // bitwise: no branch, so that the eight loads stay in flight together
      const bool ok = (e < n_stage) & (off >= 0) & (col >= CIN) & (col < (a.W + 1) * CIN);
      v[u] = *(ok ? in + off + (col - CIN) : k_conv_zero);  // staged column 0: padding
      ec.next();
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {  // past the rows: the spare float after them
      const int e = e0 + 256 * u;
      x_s[e < n_stage ? e : n_stage] = v[u];
    }
  }
  __syncthreads();
}

template <int CIN, int STRIDE>
__global__ __launch_bounds__(256) void conv_thin_wgrad_kernel(ConvArgs a) {
  extern __shared__ float x_s[];  // [range row][tap row][width][CIN]
  __shared__ float red[4][32][33];
  constexpr int N = 9 * CIN + 1;
  const int z = blockIdx.y;
  const int M = a.Co;
  const int R = thin_rows_per_range(a), wop = thin_wo_pad(a), width = thin_row_width(a);
  const int per_row = width * CIN;
  const int rows_total = a.B * a.Ho;
  const int r0 = blockIdx.x * R;
  const int nr_rows = rows_total - r0 < R ? rows_total - r0 : R;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, l32 = lane & 31, h = lane >> 5;
  thin_stage<CIN, STRIDE>(a, z, r0, R, nr_rows, per_row, x_s);
  // this lane's B column: tap (r, s) and channel c, the bias column, or none
  const int rs = l32 / CIN, nc = l32 - rs * CIN, nr = rs / 3, ns = rs - 3 * nr;
  const bool ntap = l32 < N - 1;
  const float bconst = l32 == N - 1 ? 1.0f : 0.0f;
  const int tap_off = ntap ? (nr * width + ns) * CIN + nc : 0;
  const bool mrow = l32 < M;
  const float* dz = a.dout + z * a.dout_slot;
  f32x16 acc;
#pragma unroll
  for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
  // batches of this wave: (range row q = wave + 4 (t / nj), pixel block t % nj)
  const int nj = wop / 32;
  const int my_rows = nr_rows > wave ? (nr_rows - wave + 3) / 4 : 0;
  const int nb = my_rows * nj;
  constexpr int UB = 16;
  float av[2][UB];
  auto load = [&](int t, auto P) {  // dZ of batch t (zeros past the wave's batches)
    constexpr int qs = decltype(P)::value;
    const int q = wave + 4 * (t / nj), jb = t - (t / nj) * nj;
    const bool bok = t < nb;
    const int64_t prow = static_cast<int64_t>(bok ? r0 + q : 0) * a.Wo;
    const int jlim = bok ? a.Wo - 32 * jb - h : 0;  // slots 2 u below it hold pixels
    const float* base = dz + (prow + 32 * jb + h) * M + l32;
#pragma unroll
    for (int u = 0; u < UB; ++u)
      av[qs][u] = *((mrow & (2 * u < jlim)) ? base + static_cast<int64_t>(2 * u) * M : k_conv_zero);
  };
  auto mul = [&](int t, auto P) {
    constexpr int qs = decltype(P)::value;
    const int q = wave + 4 * (t / nj), jb = t - (t / nj) * nj;
    const float* xrow = x_s + q * 3 * per_row + (STRIDE * (32 * jb + h)) * CIN + tap_off;
    float bv[UB];
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const float xv = xrow[2 * STRIDE * CIN * u];  // read by every lane (tap_off 0 past the taps)
      bv[u] = ntap ? xv : bconst;
    }
#pragma unroll
    for (int u = 0; u < UB; ++u)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av[qs][u], bv[u], acc, 0, 0, 0);
  };
  load(0, Pi<0>());
  int t = 0;
  for (; t + 1 < nb; t += 2) {
    load(t + 1, Pi<1>());
    mul(t, Pi<0>());
    load(t + 2, Pi<0>());
    mul(t + 1, Pi<1>());
  }
  if (t < nb) mul(t, Pi<0>());
  // accumulator e of lane (l32, h): row 8 (e / 4) + 4 h + e % 4, column l32
#pragma unroll
  for (int e = 0; e < 16; ++e) red[wave][8 * (e >> 2) + 4 * h + (e & 3)][l32] = acc[e];
  __syncthreads();
  for (int idx = threadIdx.x; idx < M * N; idx += 256) {
    const int m = idx / N, c = idx - m * N;
    const float v = ((red[0][m][c] + red[1][m][c]) + red[2][m][c]) + red[3][m][c];
    a.part[z * a.part_slot + (static_cast<int64_t>(blockIdx.x) * M + m) * N + c] = v;
  }
}

// Forward over whole output rows (the ranges of conv_thin_wgrad_kernel, input
// rows staged the same way): Z[p][o] = (sum over the taps of in(tap) W[o][t])
// + b[o], then ReLU, as conv_thin_fwd_kernel (same MFMA blocks and k order:
// tap j in lanes 0-31, tap J + j in lanes 32-63), but each tap is an LDS read
// at a per-lane offset fixed for the whole launch.  Wave w takes range rows
// w, w + 4, ..., each in blocks of 32 pixels.
template <int CIN, int STRIDE>
__global__ __launch_bounds__(256) void conv_thin_fwd_rows_kernel(ConvArgs a) {
  extern __shared__ float x_s[];
  constexpr int KT = 9 * CIN, J = (KT + 1) / 2;
  const int z = blockIdx.y;
  const int R = thin_rows_per_range(a, THIN_FWD_PIXELS), wop = thin_wo_pad(a);
  const int width = thin_row_width(a);
  const int per_row = width * CIN;
  const int rows_total = a.B * a.Ho;
  const int r0 = blockIdx.x * R;
  const int nr_rows = rows_total - r0 < R ? rows_total - r0 : R;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, l32 = lane & 31, h = lane >> 5;
  const float* par = a.master_in + static_cast<int64_t>(a.order[z]) * a.master_in_slot;
  const bool col_ok = l32 < a.Co;
  float wv[J];
  int toff[J];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int t = j + J * h;
    wv[j] = *(col_ok && t < KT ? par + a.w_off + static_cast<int64_t>(l32) * KT + t
                               : k_conv_zero);
    const int rs = h ? tap_rs(j + J, CIN) : tap_rs(j, CIN);
    const int c = h ? tap_c(j + J, CIN) : tap_c(j, CIN);
    const int r = rs / 3, sc = rs - 3 * r;
    toff[j] = t < KT ? (r * width + sc) * CIN + c : 0;  // padding taps have zero weights
  }
  const float bias = *(col_ok ? par + a.b_off + l32 : k_conv_zero);
  thin_stage<CIN, STRIDE>(a, z, r0, R, nr_rows, per_row, x_s);
  const int nj = wop / 32;
  const int my_rows = nr_rows > wave ? (nr_rows - wave + 3) / 4 : 0;
  float* out = a.out + z * a.out_slot;
  for (int t = 0; t < my_rows * nj; ++t) {
    const int q = wave + 4 * (t / nj), jb = t - (t / nj) * nj;
    const float* xp = x_s + q * 3 * per_row + STRIDE * (32 * jb + l32) * CIN;
    float xv[J];
#pragma unroll
    for (int j = 0; j < J; ++j) xv[j] = xp[toff[j]];
    f32x16 acc;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
#pragma unroll
    for (int j = 0; j < J; ++j) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(xv[j], wv[j], acc, 0, 0, 0);
    // accumulator e of lane (l32, h): pixel 8 (e / 4) + 4 h + e % 4 of the block, channel l32
    const int jlim = a.Wo - 32 * jb;
    float* orow = out + (static_cast<int64_t>(r0 + q) * a.Wo + 32 * jb) * a.Co + l32;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int pj = 8 * (e >> 2) + 4 * h + (e & 3);
      const float v = acc[e] + bias;
      if ((pj < jlim) & col_ok) orow[pj * a.Co] = v > 0.0f ? v : 0.0f;
    }
  }
}

// All SGD updates of one local step in one launch, after every layer's
// backward-data has read its weights.  Block j of u is a layer's weights
// W[m][n] (n < N - 1) and bias b[m] (n = N - 1); a workgroup takes UW
// consecutive weights of one block.  The gradient of weight (m, n) is
//   with partials (a weight-gradient launch's ranges): the sum of the
//     ranges' partials in UG groups of consecutive ranges, each group in
//     range order by one thread (sixteen partials loaded at a time), then
//     the group sums in group order;
//   without (the classifier after conv_head_kernel): the sum over the batch
//     of delta[b][m] pooled[b][n] (pooled = 1 for the bias) in UG groups of
//     consecutive rows, each in row order, then the group sums in order.
// The order depends on the sizes only, not on how many replicas share the
// launch.  master[order[z]] <- master_in[order[z]] - lr (gradient).
constexpr int UW = 32, UG = 8;
static_assert(UW * UG == 256, "one thread per (weight, group)");

struct UpdateAll {
  UpdateBlock blk[MAX_UPDATE_BLOCKS];
  int64_t first[MAX_UPDATE_BLOCKS + 1];  // first workgroup of each block
  int n;
  const float* master_in;
  int64_t master_in_slot;
  const int32_t* order;
};

__global__ __launch_bounds__(256) void conv_update_all_kernel(UpdateAll u, HeadArgs h,
                                                              float* master, int64_t master_slot,
                                                              float lr) {
  int j = 0;
  while (j + 1 < u.n && blockIdx.x >= u.first[j + 1]) ++j;
  const UpdateBlock ub = u.blk[j];
  const int z = blockIdx.y;
  const int rep = u.order[z];
  const int64_t MN = static_cast<int64_t>(ub.M) * ub.N;
  const int w = threadIdx.x % UW, grp = threadIdx.x / UW;
  const int64_t e = (static_cast<int64_t>(blockIdx.x) - u.first[j]) * UW + w;
  const int64_t m = e / ub.N, n = e - m * ub.N;
  float sum = 0.0f;
  if (e < MN) {
    if (ub.part) {
      const int per = (ub.splits + UG - 1) / UG;
      const int s0 = grp * per, s1 = min(ub.splits, s0 + per);
      const float* part = ub.part + z * ub.part_slot;
      int sp = s0;
      for (; sp + 16 <= s1; sp += 16) {
        float v[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) v[q] = part[(sp + q) * MN + e];
#pragma unroll
        for (int q = 0; q < 16; ++q) sum += v[q];
      }
      for (; sp < s1; ++sp) sum += part[sp * MN + e];
    } else {
      const int per = (h.B + UG - 1) / UG;
      const int b0 = grp * per, b1 = min(h.B, b0 + per);
      const float* dcol = h.delta + z * h.delta_slot + m;
      // the bias column reads ones
      const float* pcol = n < ub.N - 1 ? h.pooled + z * h.pooled_slot + n : k_conv_one;
      const int64_t ps = n < ub.N - 1 ? ub.N - 1 : 0;
      int bb = b0;
      for (; bb + 8 <= b1; bb += 8) {
        float dv[8], pv[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          dv[q] = dcol[static_cast<int64_t>(bb + q) * h.delta_ld];
          pv[q] = pcol[(bb + q) * ps];
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) sum = fmaf(dv[q], pv[q], sum);
      }
      for (; bb < b1; ++bb)
        sum = fmaf(dcol[static_cast<int64_t>(bb) * h.delta_ld], pcol[bb * ps], sum);
    }
  }
  __shared__ float group_sum[UG][UW];
  group_sum[grp][w] = sum;
  __syncthreads();
  if (grp != 0 || e >= MN) return;
  float tot = group_sum[0][w];
#pragma unroll
  for (int g = 1; g < UG; ++g) tot += group_sum[g][w];
  const float* src = u.master_in + static_cast<int64_t>(rep) * u.master_in_slot;
  float* dst = master + static_cast<int64_t>(rep) * master_slot;
  const int64_t at = n < ub.N - 1 ? ub.w_off + m * (ub.N - 1) + n : ub.b_off + m;
  dst[at] = fmaf(-lr, tot, src[at]);
}

// pooled[b][c] = (sum over the positions) / (H W): the positions in PG groups
// of consecutive positions, each in position order by one thread, then the
// group sums in group order.  A workgroup takes PW consecutive channels of one
// batch row (a half-wave's loads read consecutive channels of one position).
constexpr int PW = 32, PG = 8;
static_assert(PW * PG == 256, "one thread per (channel, group)");

__global__ __launch_bounds__(256) void avgpool_kernel(const float* act, int64_t act_slot,
                                                      float* pooled, int64_t pooled_slot, int B,
                                                      int HW, int C) {
  const int z = blockIdx.y;
  const int cb = (C + PW - 1) / PW;
  const int b = blockIdx.x / cb, c = (blockIdx.x % cb) * PW + threadIdx.x % PW;
  const int grp = threadIdx.x / PW;
  const int per = (HW + PG - 1) / PG;
  const int p0 = grp * per, p1 = min(HW, p0 + per);
  float sum = 0.0f;
  if (c < C) {
    const float* src = act + z * act_slot + (static_cast<int64_t>(b) * HW) * C + c;
    for (int p = p0; p < p1; ++p) sum += src[static_cast<int64_t>(p) * C];
  }
  __shared__ float group_sum[PG][PW];
  group_sum[grp][threadIdx.x % PW] = sum;
  __syncthreads();
  if (grp != 0 || c >= C) return;
  float tot = group_sum[0][threadIdx.x];
#pragma unroll
  for (int g = 1; g < PG; ++g) tot += group_sum[g][threadIdx.x];
  pooled[z * pooled_slot + static_cast<int64_t>(b) * C + c] = tot / static_cast<float>(HW);
}

__global__ __launch_bounds__(256) void avgpool_backward_kernel(const float* dpooled,
                                                               int64_t dpooled_slot,
                                                               const float* act, int64_t act_slot,
                                                               float* dz, int B, int HW, int C) {
  const int z = blockIdx.y;
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t per = static_cast<int64_t>(B) * HW * C;
  if (e >= per) return;
  const int64_t b = e / (static_cast<int64_t>(HW) * C), c = e % C;
  const float g = dpooled[z * dpooled_slot + b * C + c] / static_cast<float>(HW);
  dz[z * act_slot + e] = act[z * act_slot + e] > 0.0f ? g : 0.0f;
}

// The classifier head of one batch row b of slot z in one workgroup: the
// row's last conv activation act[b] is staged in LDS once and serves the
// pooling and the ReLU mask of the pooling backward.
//   pooled[c] = (sum over the positions p, in order, of act[p][c]) / HW
//   logit[o] = bias[o] + sum_c pooled[c] W[o][c]  (one wave per class: each
//              lane over its channels c = lane, lane + 64, ..., then an
//              xor-butterfly over the lanes)
//   softmax cross-entropy as softmax_ce_kernel: loss = log(sum_o exp(logit[o]
//   - max)) - (logit[label] - max); delta[o] = (softmax[o] - [o = label]) / B
//   dz[p][c] = (sum over o, in order, of delta[o] W[o][c]) / HW where
//              act[p][c] > 0, else 0
// LDS: HW C + 2 C + classes floats.
constexpr int HEAD_LDS_FLOATS = 12288;

__device__ __forceinline__ float wave_sum(float v) {
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
  for (int d = 32; d >= 1; d >>= 1) v = fmaxf(v, __shfl_xor(v, d));
  return v;
}

__global__ __launch_bounds__(256) void conv_head_kernel(HeadArgs h) {
  extern __shared__ float head_s[];
  const int z = blockIdx.y, b = blockIdx.x, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = h.HW * h.C;
  float* a_s = head_s;               // act[b], n floats
  float* pool_s = a_s + n;           // C
  float* dp_s = pool_s + h.C;        // C
  float* lg_s = dp_s + h.C;          // classes: logits, then delta
  const float* act_b = h.act + z * h.act_slot + static_cast<int64_t>(b) * n;
  const bool vec = (n & 3) == 0 && (reinterpret_cast<uintptr_t>(act_b) & 15) == 0;
  if (vec) {
    for (int i = 4 * tid; i < n; i += 1024)
      *reinterpret_cast<f32x4*>(a_s + i) = *reinterpret_cast<const f32x4*>(act_b + i);
  } else {
    for (int i = tid; i < n; i += 256) a_s[i] = act_b[i];
  }
  __syncthreads();
  const float inv_hw = 1.0f / static_cast<float>(h.HW);
  for (int c = tid; c < h.C; c += 256) {
    float sum = 0.0f;
    for (int p = 0; p < h.HW; ++p) sum += a_s[p * h.C + c];
    const float v = sum / static_cast<float>(h.HW);
    pool_s[c] = v;
    h.pooled[z * h.pooled_slot + static_cast<int64_t>(b) * h.C + c] = v;
  }
  __syncthreads();
  const float* par = h.master_in + static_cast<int64_t>(h.order[z]) * h.master_in_slot;
  const float* Wc = par + h.w_off;
  for (int o = wave; o < h.classes; o += 4) {
    float v = 0.0f;
    for (int c = lane; c < h.C; c += 64) v = fmaf(pool_s[c], Wc[static_cast<int64_t>(o) * h.C + c], v);
    v = wave_sum(v);
    if (lane == 0) lg_s[o] = par[h.b_off + o] + v;
  }
  __syncthreads();
  if (wave == 0) {
    const int label = h.y[h.gather[z * h.gather_slot + b]];
    const bool label_ok = label >= 0 && label < h.classes;
    float mx = -INFINITY;
    for (int o = lane; o < h.classes; o += 64) mx = fmaxf(mx, lg_s[o]);
    mx = wave_max(mx);
    float sum = 0.0f;
    for (int o = lane; o < h.classes; o += 64) sum += expf(lg_s[o] - mx);
    sum = wave_sum(sum);
    const float zl = label_ok ? lg_s[label] : 0.0f;
    const float invB = 1.0f / static_cast<float>(h.B);
    float* drow = h.delta + z * h.delta_slot + static_cast<int64_t>(b) * h.delta_ld;
    for (int o = lane; o < h.delta_ld; o += 64) {
      float dv = 0.0f;
      if (o < h.classes) {
        dv = (expf(lg_s[o] - mx) / sum - (o == label ? 1.0f : 0.0f)) * invB;
        lg_s[o] = dv;
      }
      drow[o] = dv;
    }
    if (lane == 0)
      h.loss[z * h.loss_slot + b] = label_ok ? logf(sum) - (zl - mx) : __builtin_nanf("");
  }
  __syncthreads();
  for (int c = tid; c < h.C; c += 256) {
    float v = 0.0f;
    for (int o = 0; o < h.classes; ++o) v = fmaf(lg_s[o], Wc[static_cast<int64_t>(o) * h.C + c], v);
    dp_s[c] = v * inv_hw;
  }
  __syncthreads();
  float* dz_b = h.dz + z * h.dz_slot + static_cast<int64_t>(b) * n;
  if (vec && (h.C & 3) == 0 && (reinterpret_cast<uintptr_t>(dz_b) & 15) == 0) {
    for (int i = 4 * tid; i < n; i += 1024) {
      const int c = i % h.C;
      const f32x4 av = *reinterpret_cast<const f32x4*>(a_s + i);
      f32x4 g;
#pragma unroll
      for (int e = 0; e < 4; ++e) g[e] = av[e] > 0.0f ? dp_s[c + e] : 0.0f;
      *reinterpret_cast<f32x4*>(dz_b + i) = g;
    }
  } else {
    for (int i = tid; i < n; i += 256) dz_b[i] = a_s[i] > 0.0f ? dp_s[i % h.C] : 0.0f;
  }
}

int conv_cu_count() {
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


// Launches of at most two workgroups per CU (one or two replicas) take K
// steps of 32 (one barrier per 16 MFMAs instead of 8): with one or two waves
// per SIMD nothing else hides a step's fixed cost.  With the vector loaders
// only (the general gathers spill with two halves).
template <int PASS, bool TR>
void launch_conv_gemm(const dim3& grid, hipStream_t s, const ConvArgs& a) {
  const int64_t wgs = static_cast<int64_t>(grid.x) * grid.y;
  const bool wide = wgs <= 2LL * conv_cu_count();
  if constexpr (PASS == CONV_WGRAD && TR) {
    if (a.gather) {  // gathered dataset rows (a first layer with four or more channels)
      hipLaunchKernelGGL((conv_gemm_kernel<PASS, TR, 1, true>), grid, dim3(256), 0, s, a);
      return;
    }
  }
  if constexpr (TR) {
    if (wide) {
      hipLaunchKernelGGL((conv_gemm_kernel<PASS, TR, 2>), grid, dim3(256), 0, s, a);
      return;
    }
  }
  hipLaunchKernelGGL((conv_gemm_kernel<PASS, TR, 1>), grid, dim3(256), 0, s, a);
}

}  // namespace

hipError_t launch_conv(const ConvArgs& a, ConvPass pass, int n_slots, hipStream_t s) {
  // shortcuts: conv forward and backward-data on the 64 x 64 and narrow tiles only
  if (a.skip && (pass == FC_FWD || pass == FC_DGRAD || pass == CONV_WGRAD || pass == FC_WGRAD ||
                 (pass == CONV_FWD && thin_layer(a))))
    return hipErrorInvalidValue;
  if (pass == CONV_DGRAD && dgrad_narrow(a)) {
    if (n_slots < 1 || a.cls > 3 || a.B < 1 || a.Co < 1 || (a.stride == 2 && a.cls < -1))
      return hipErrorInvalidValue;
    int64_t gx = 0;
    if (a.stride == 2 && a.cls < 0) {
      for (int i = 0; i < 4; ++i) {
        ConvArgs ac = a;
        ac.cls = i;
        gx += dgrad_narrow_tiles(ac);
      }
    } else {
      gx = dgrad_narrow_tiles(a);
    }
    if (gx == 0) return hipSuccess;  // no pixels (extents of 1)
    if (gx > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(conv_dgrad_narrow_kernel, dim3(static_cast<unsigned>(gx), n_slots),
                       dim3(256), 0, s, a);
    return hipGetLastError();
  }
  if (pass == CONV_DGRAD && a.stride == 2) {
    if (n_slots < 1 || a.cls > 3 || a.B < 1 || a.C < 1 || a.Co < 1) return hipErrorInvalidValue;
    int64_t gx = 0;
    if (a.cls < 0)
      for (int i = 0; i < 4; ++i) gx += dgrad_class_tiles(a, i);
    else
      gx = dgrad_class_tiles(a, a.cls);
    if (gx == 0) return hipSuccess;  // no pixels (extents of 1)
    if (gx > 0x7FFFFFFF) return hipErrorInvalidValue;
    if (vector_loaders(a))
      launch_conv_gemm<CONV_DGRAD, true>(dim3(static_cast<unsigned>(gx), n_slots), s, a);
    else
      launch_conv_gemm<CONV_DGRAD, false>(dim3(static_cast<unsigned>(gx), n_slots), s, a);
    return hipGetLastError();
  }
  const Dims d = pass_dims(a, pass);
  if (n_slots < 1 || d.M < 1 || d.N < 1 || d.K < 1) return hipErrorInvalidValue;
  if (pass == CONV_FWD && thin_wgrad(a)) {
    const int R = thin_rows_per_range(a, THIN_FWD_PIXELS);
    const dim3 grid(static_cast<unsigned>((a.B * a.Ho + R - 1) / R), n_slots), block(256);
    // staged rows and one spare float (the target of stores past the rows)
    const size_t lds = static_cast<size_t>(thin_stage_floats(a, THIN_FWD_PIXELS) + 1) * sizeof(float);
    switch (2 * a.C + (a.stride == 2 ? 1 : 0)) {
      case 2: hipLaunchKernelGGL((conv_thin_fwd_rows_kernel<1, 1>), grid, block, lds, s, a); break;
      case 3: hipLaunchKernelGGL((conv_thin_fwd_rows_kernel<1, 2>), grid, block, lds, s, a); break;
      case 4: hipLaunchKernelGGL((conv_thin_fwd_rows_kernel<2, 1>), grid, block, lds, s, a); break;
      case 5: hipLaunchKernelGGL((conv_thin_fwd_rows_kernel<2, 2>), grid, block, lds, s, a); break;
      case 6: hipLaunchKernelGGL((conv_thin_fwd_rows_kernel<3, 1>), grid, block, lds, s, a); break;
      default: hipLaunchKernelGGL((conv_thin_fwd_rows_kernel<3, 2>), grid, block, lds, s, a); break;
    }
    return hipGetLastError();
  }
  if (pass == CONV_FWD && thin_layer(a)) {
    const int64_t blocks = (d.M + 4 * 32 * THIN_TB - 1) / (4 * 32 * THIN_TB);
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(blocks), n_slots), block(256);
    switch (a.C) {
      case 1: hipLaunchKernelGGL(conv_thin_fwd_kernel<1>, grid, block, 0, s, a); break;
      case 2: hipLaunchKernelGGL(conv_thin_fwd_kernel<2>, grid, block, 0, s, a); break;
      default: hipLaunchKernelGGL(conv_thin_fwd_kernel<3>, grid, block, 0, s, a); break;
    }
    return hipGetLastError();
  }
  if (pass == CONV_WGRAD && thin_wgrad(a)) {
    const int R = thin_rows_per_range(a);
    if (a.k_per_split != R || a.splits != (a.B * a.Ho + R - 1) / R) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(a.splits), n_slots), block(256);
    const size_t lds = static_cast<size_t>(thin_stage_floats(a) + 1) * sizeof(float);
    const int key = 2 * a.C + (a.stride == 2 ? 1 : 0);
    switch (key) {
      case 2: hipLaunchKernelGGL((conv_thin_wgrad_kernel<1, 1>), grid, block, lds, s, a); break;
      case 3: hipLaunchKernelGGL((conv_thin_wgrad_kernel<1, 2>), grid, block, lds, s, a); break;
      case 4: hipLaunchKernelGGL((conv_thin_wgrad_kernel<2, 1>), grid, block, lds, s, a); break;
      case 5: hipLaunchKernelGGL((conv_thin_wgrad_kernel<2, 2>), grid, block, lds, s, a); break;
      case 6: hipLaunchKernelGGL((conv_thin_wgrad_kernel<3, 1>), grid, block, lds, s, a); break;
      default: hipLaunchKernelGGL((conv_thin_wgrad_kernel<3, 2>), grid, block, lds, s, a); break;
    }
    return hipGetLastError();
  }
  if (pass == CONV_FWD && conv_narrow(a)) {
    const int64_t gx = fwd_narrow_tiles(a);
    if (gx > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(conv_fwd_narrow_kernel, dim3(static_cast<unsigned>(gx), n_slots), dim3(256),
                       0, s, a);
    return hipGetLastError();
  }
  if (pass == CONV_WGRAD && conv_narrow(a)) {
    if (a.splits < 1 || a.k_per_split < 1 ||
        static_cast<int64_t>(a.splits) * a.k_per_split < d.K)
      return hipErrorInvalidValue;
    const int64_t gx = wgrad_narrow_tiles(a) * a.splits;
    if (gx > 0x7FFFFFFF) return hipErrorInvalidValue;
    if (a.gather)
      hipLaunchKernelGGL(conv_wgrad_narrow_kernel<true>, dim3(static_cast<unsigned>(gx), n_slots),
                         dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL(conv_wgrad_narrow_kernel<false>, dim3(static_cast<unsigned>(gx), n_slots),
                         dim3(256), 0, s, a);
    return hipGetLastError();
  }
  int64_t gx = ((d.M + CT - 1) / CT) * ((d.N + CT - 1) / CT);
  if (pass == CONV_WGRAD || pass == FC_WGRAD) {
    if (a.splits < 1 || a.k_per_split < 1 ||
        static_cast<int64_t>(a.splits) * a.k_per_split < d.K)
      return hipErrorInvalidValue;
    gx *= a.splits;
  }
  if (gx > 0x7FFFFFFF) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(gx), n_slots), block(256);
  switch (pass) {
    case CONV_FWD:
      if (vector_loaders(a))
        launch_conv_gemm<CONV_FWD, true>(grid, s, a);
      else
        launch_conv_gemm<CONV_FWD, false>(grid, s, a);
      break;
    case CONV_DGRAD:
      if (vector_loaders(a))
        launch_conv_gemm<CONV_DGRAD, true>(grid, s, a);
      else
        launch_conv_gemm<CONV_DGRAD, false>(grid, s, a);
      break;
    case CONV_WGRAD:
      if (vector_loaders(a))
        launch_conv_gemm<CONV_WGRAD, true>(grid, s, a);
      else
        launch_conv_gemm<CONV_WGRAD, false>(grid, s, a);
      break;
    case FC_FWD: launch_conv_gemm<FC_FWD, false>(grid, s, a); break;
    case FC_DGRAD: launch_conv_gemm<FC_DGRAD, false>(grid, s, a); break;
    case FC_WGRAD: launch_conv_gemm<FC_WGRAD, false>(grid, s, a); break;
  }
  return hipGetLastError();
}

namespace {
// Tiles of the two launches conv_bwd_pair_kernel joins, or false where it
// does not apply (channel counts for the vector loaders, no gathered rows).
// Joined at every replica count: on the CIFAR-shaped networks of 3 and 9
// conv layers (K = 8) a round took 2.65 / 14.4 ms, against 2.67 / 14.6 ms with
// the pair only up to twelve workgroups per CU and 2.75 / 15.2 ms with two
// launches everywhere.
bool conv_pair_plan(const ConvArgs& d, const ConvArgs& w, int n_slots, bool* dn, bool* wn,
                    int64_t* nd, int64_t* nw) {
  if (n_slots < 1 || !vector_loaders(d) || !vector_loaders(w) || d.gather || w.gather ||
      thin_layer(w) || d.B < 1 || d.cls > 3 || (d.stride == 2 && d.cls < -1) || w.splits < 1 ||
      w.k_per_split < 1)
    return false;
  const Dims dw = pass_dims(w, CONV_WGRAD);
  if (static_cast<int64_t>(w.splits) * w.k_per_split < dw.K) return false;
  *dn = dgrad_narrow(d);
  int64_t t = 0;
  const bool all = d.stride == 2 && d.cls < 0;
  for (int i = 0; i < (all ? 4 : 1); ++i) {
    ConvArgs ac = d;
    if (all) ac.cls = i;
    if (*dn) {
      t += dgrad_narrow_tiles(ac);
    } else if (d.stride == 2) {
      t += dgrad_class_tiles(ac, ac.cls);
    } else {
      const Dims dd = pass_dims(ac, CONV_DGRAD);
      t += ((dd.M + CT - 1) / CT) * ((dd.N + CT - 1) / CT);
    }
  }
  *nd = t;
  *wn = conv_narrow(w);
  *nw = (*wn ? wgrad_narrow_tiles(w) : ((dw.M + CT - 1) / CT) * ((dw.N + CT - 1) / CT)) * w.splits;
  return *nd > 0 && *nw > 0 && *nd + *nw <= 0x7FFFFFFF;
}
}  // namespace

bool conv_pair_fits(const ConvArgs& d, const ConvArgs& w, int n_slots) {
  bool dn, wn;
  int64_t nd, nw;
  return conv_pair_plan(d, w, n_slots, &dn, &wn, &nd, &nw);
}

hipError_t launch_conv_pair(const ConvArgs& d, const ConvArgs& w, int n_slots, hipStream_t s) {
  bool dn, wn;
  int64_t nd, nw;
  if (!conv_pair_plan(d, w, n_slots, &dn, &wn, &nd, &nw)) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(nd + nw), n_slots), block(256);
  const int ndi = static_cast<int>(nd);
  if (dn && wn)
    hipLaunchKernelGGL((conv_bwd_pair_kernel<true, true>), grid, block, 0, s, d, w, ndi);
  else if (dn)
    hipLaunchKernelGGL((conv_bwd_pair_kernel<true, false>), grid, block, 0, s, d, w, ndi);
  else if (wn)
    hipLaunchKernelGGL((conv_bwd_pair_kernel<false, true>), grid, block, 0, s, d, w, ndi);
  else
    hipLaunchKernelGGL((conv_bwd_pair_kernel<false, false>), grid, block, 0, s, d, w, ndi);
  return hipGetLastError();
}

hipError_t launch_conv_updates(const UpdateBlock* blocks, int n_blocks, const HeadArgs* head,
                               const float* master_in, int64_t master_in_slot, const int32_t* order,
                               float* master, int64_t master_slot, float lr, int n_slots,
                               hipStream_t s) {
  if (n_blocks < 1 || n_blocks > MAX_UPDATE_BLOCKS || n_slots < 1) return hipErrorInvalidValue;
  UpdateAll u{};
  u.n = n_blocks;
  u.master_in = master_in;
  u.master_in_slot = master_in_slot;
  u.order = order;
  HeadArgs h{};
  int64_t total = 0;
  for (int j = 0; j < n_blocks; ++j) {
    const UpdateBlock& b = blocks[j];
    if (b.M < 1 || b.N < 2) return hipErrorInvalidValue;
    if (b.part ? b.splits < 1 : (!head || head->B < 1 || head->classes != b.M || head->C + 1 != b.N))
      return hipErrorInvalidValue;
    u.blk[j] = b;
    u.first[j] = total;
    total += (static_cast<int64_t>(b.M) * b.N + UW - 1) / UW;
  }
  u.first[n_blocks] = total;
  if (head) h = *head;
  if (total > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(conv_update_all_kernel, dim3(static_cast<unsigned>(total), n_slots),
                     dim3(256), 0, s, u, h, master, master_slot, lr);
  return hipGetLastError();
}

hipError_t launch_avgpool(const float* act, int64_t act_slot, float* pooled, int64_t pooled_slot,
                          int B, int HW, int C, int n_slots, hipStream_t s) {
  const int64_t blocks = static_cast<int64_t>(B) * ((C + PW - 1) / PW);
  if (blocks > 0x7FFFFFFF || n_slots < 1 || B < 1 || HW < 1 || C < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(avgpool_kernel, dim3(static_cast<unsigned>(blocks), n_slots), dim3(256), 0, s,
                     act, act_slot, pooled, pooled_slot, B, HW, C);
  return hipGetLastError();
}

hipError_t launch_avgpool_backward(const float* dpooled, int64_t dpooled_slot, const float* act,
                                   int64_t act_slot, float* dz, int B, int HW, int C,
                                   int n_slots, hipStream_t s) {
  const int64_t blocks = (static_cast<int64_t>(B) * HW * C + 255) / 256;
  if (blocks > 0x7FFFFFFF || n_slots < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(avgpool_backward_kernel, dim3(static_cast<unsigned>(blocks), n_slots),
                     dim3(256), 0, s, dpooled, dpooled_slot, act, act_slot, dz, B, HW, C);
  return hipGetLastError();
}

bool conv_head_fits(int HW, int C, int classes) {
  if (HW < 1 || C < 1 || classes < 1) return false;
  const int64_t need = static_cast<int64_t>(HW) * C + 2LL * C + classes;
  return need <= HEAD_LDS_FLOATS;
}

hipError_t launch_conv_head(const HeadArgs& h, int n_slots, hipStream_t s) {
  if (n_slots < 1 || h.B < 1 || !conv_head_fits(h.HW, h.C, h.classes) || h.delta_ld < h.classes)
    return hipErrorInvalidValue;
  const size_t lds = (static_cast<size_t>(h.HW) * h.C + 2 * h.C + h.classes) * sizeof(float);
  hipLaunchKernelGGL(conv_head_kernel, dim3(static_cast<unsigned>(h.B), n_slots), dim3(256), lds, s,
                     h);
  return hipGetLastError();
}

void conv_wgrad_ranges(const ConvArgs& a, int* splits, int64_t* k_per_split) {
  if (thin_wgrad(a)) {
    const int R = thin_rows_per_range(a);
    *k_per_split = R;
    *splits = (a.B * a.Ho + R - 1) / R;
    return;
  }
  const int64_t pixels = static_cast<int64_t>(a.B) * a.Ho * a.Wo;
  *k_per_split = CONV_WGRAD_PIXELS;
  *splits = static_cast<int>((pixels + CONV_WGRAD_PIXELS - 1) / CONV_WGRAD_PIXELS);
}

}  // namespace oscars
