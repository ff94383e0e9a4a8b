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
// Backward-data of a stride-2 layer runs one launch per parity class of the
// input pixels: input row hi receives output row i through tap r only where
// hi + 1 - r = 2 i, so even rows take tap r = 1 and odd rows taps 0 and 2
// (likewise columns).  Each class gathers only its 1, 2 or 4 taps (K = taps x
// Cout), a quarter of the 9-tap work on average.
// A workgroup computes a 64 x 64 tile of C with four waves of 32 x 32, fp32
// MFMA 32x32x2, K in steps of 16: the next step's operands are gathered into
// registers while the current step's MFMAs read LDS (two LDS buffers, one
// barrier per step).  The weight-gradient passes split K into ranges, one
// partial sum per range, which the update kernel adds in range order before
// applying the SGD step of Eq. 4 -- so results depend on nothing but the
// inputs, whichever slots share a launch.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "conv.h"

namespace oscars {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int CT = 64;       // tile rows and columns
constexpr int CK = 16;       // K per step
constexpr int CLD = CT + 4;  // LDS row pitch (floats)

struct Dims {
  int64_t M, N, K;
};

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

  // Kernel tap (r, s) of backward-data tap index t: all nine (t = 3 r + s)
  // for stride 1; the class's one, two or four for stride 2.
  __device__ __forceinline__ void dgrad_tap_rs(int t, int& r, int& s) const {
    if (a.stride == 2) {
      const int ns = cls_taps(a.cls & 1), tr = t / ns, ts = t - tr * ns;
      r = (a.cls >> 1) ? 2 * tr : 1;
      s = (a.cls & 1) ? 2 * ts : 1;
    } else {
      r = t / 3;
      s = t - 3 * r;
    }
  }

  __device__ __forceinline__ const float* image(int b) const {
    return rows ? in + static_cast<int64_t>(rows[b]) * a.in_ld
                : in + static_cast<int64_t>(b) * a.H * a.W * a.C;
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

template <int PASS>
__global__ __launch_bounds__(256) void conv_gemm_kernel(ConvArgs a) {
  constexpr bool WG = PASS == CONV_WGRAD || PASS == FC_WGRAD;
  __shared__ float As[2][CK][CLD];
  __shared__ float Bs[2][CK][CLD];
  const Dims d = pass_dims(a, PASS);
  const int M = static_cast<int>(d.M), N = static_cast<int>(d.N), K = static_cast<int>(d.K);
  const int z = blockIdx.y;
  const int rep = a.order[z];
  const int gm = (M + CT - 1) / CT, gn = (N + CT - 1) / CT;
  int tile = blockIdx.x, split = 0;
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
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  const ConvLoader<PASS> ld(a, kend, m0 + lr, M, n0 + lr, N, in, rows, dz, par + a.w_off);
  float ra[4], rb[4];
  auto stash = [&](int buf) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      As[buf][lk + e][lr] = ra[e];
      Bs[buf][lk + e][lr] = rb[e];
    }
  };

  f32x16 acc;
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.0f;
  const int nk = (kend - kbeg + CK - 1) / CK;
  ld.fetch(kbeg + lk, ra, rb);
  stash(0);
  __syncthreads();
  for (int t = 0; t < nk; ++t) {
    const int buf = t & 1;
    if (t + 1 < nk) ld.fetch(kbeg + (t + 1) * CK + lk, ra, rb);
    // MFMA u contracts k = 2u (lanes 0-31) and 2u + 1 (lanes 32-63)
#pragma unroll
    for (int u = 0; u < CK / 2; ++u)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(As[buf][2 * u + h][wm * 32 + r],
                                                 Bs[buf][2 * u + h][wn * 32 + r], acc, 0, 0, 0);
    if (t + 1 < nk) stash(buf ^ 1);
    __syncthreads();
  }

  // accumulator i of lane (r, h): row 8 (i / 4) + 4 h + i % 4, column r
  const int col = n0 + wn * 32 + r;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int row = m0 + wm * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
    if (row >= M || col >= N) continue;
    const float v = acc[i];
    if constexpr (PASS == CONV_FWD) {
      const float zv = v + par[a.b_off + col];
      a.out[z * a.out_slot + static_cast<int64_t>(row) * a.Co + col] = zv > 0.0f ? zv : 0.0f;
    } else if constexpr (PASS == FC_FWD) {
      a.out[z * a.out_slot + static_cast<int64_t>(row) * a.out_ld + col] = v + par[a.b_off + col];
    } else if constexpr (PASS == CONV_DGRAD) {
      int b, hi, wi;
      ConvLoader<PASS>::dgrad_pixel(a, row, b, hi, wi);
      const int64_t at = ((static_cast<int64_t>(b) * a.H + hi) * a.W + wi) * a.C + col;
      a.out[z * a.out_slot + at] = a.mask[z * a.mask_slot + at] > 0.0f ? v : 0.0f;
    } else if constexpr (PASS == FC_DGRAD) {
      a.out[z * a.out_slot + static_cast<int64_t>(row) * a.out_ld + col] = v;
    } else {
      a.part[z * a.part_slot + (static_cast<int64_t>(split) * M + row) * N + col] = v;
    }
  }
}

// Sum of the partials of weight (m, n) in split order, then
// master <- master_in - lr sum: W[m][n] for n < N - 1, the bias b[m] for the
// last column.
template <int PASS>
__global__ __launch_bounds__(256) void conv_update_kernel(ConvArgs a, float* master,
                                                          int64_t master_slot, float lr) {
  const Dims d = pass_dims(a, PASS);
  const int z = blockIdx.y;
  const int rep = a.order[z];
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= d.M * d.N) return;
  const int64_t m = e / d.N, n = e % d.N;
  const float* part = a.part + z * a.part_slot;
  float sum = 0.0f;
  for (int s = 0; s < a.splits; ++s) sum += part[s * d.M * d.N + e];
  const float* src = a.master_in + static_cast<int64_t>(rep) * a.master_in_slot;
  float* dst = master + static_cast<int64_t>(rep) * master_slot;
  const int64_t at = n < d.N - 1 ? a.w_off + m * (d.N - 1) + n : a.b_off + m;
  dst[at] = fmaf(-lr, sum, src[at]);
}

__global__ __launch_bounds__(256) void avgpool_kernel(const float* act, int64_t act_slot,
                                                      float* pooled, int64_t pooled_slot, int B,
                                                      int HW, int C) {
  const int z = blockIdx.y;
  const int64_t e = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (e >= static_cast<int64_t>(B) * C) return;
  const int64_t b = e / C, c = e % C;
  const float* src = act + z * act_slot + b * HW * C + c;
  float sum = 0.0f;
  for (int p = 0; p < HW; ++p) sum += src[static_cast<int64_t>(p) * C];
  pooled[z * pooled_slot + e] = sum / static_cast<float>(HW);
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

}  // namespace

hipError_t launch_conv(const ConvArgs& a, ConvPass pass, int n_slots, hipStream_t s) {
  const Dims d = pass_dims(a, pass);
  if (pass == CONV_DGRAD && a.stride == 2 && d.M == 0 && n_slots >= 1)
    return hipSuccess;  // a parity class without pixels (an extent of 1)
  if (n_slots < 1 || d.M < 1 || d.N < 1 || d.K < 1) return hipErrorInvalidValue;
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
    case CONV_FWD: hipLaunchKernelGGL(conv_gemm_kernel<CONV_FWD>, grid, block, 0, s, a); break;
    case CONV_DGRAD: hipLaunchKernelGGL(conv_gemm_kernel<CONV_DGRAD>, grid, block, 0, s, a); break;
    case CONV_WGRAD: hipLaunchKernelGGL(conv_gemm_kernel<CONV_WGRAD>, grid, block, 0, s, a); break;
    case FC_FWD: hipLaunchKernelGGL(conv_gemm_kernel<FC_FWD>, grid, block, 0, s, a); break;
    case FC_DGRAD: hipLaunchKernelGGL(conv_gemm_kernel<FC_DGRAD>, grid, block, 0, s, a); break;
    case FC_WGRAD: hipLaunchKernelGGL(conv_gemm_kernel<FC_WGRAD>, grid, block, 0, s, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_conv_update(const ConvArgs& a, ConvPass pass, float* master,
                              int64_t master_slot, float lr, int n_slots, hipStream_t s) {
  if (pass != CONV_WGRAD && pass != FC_WGRAD) return hipErrorInvalidValue;
  const Dims d = pass_dims(a, pass);
  const int64_t blocks = (d.M * d.N + 255) / 256;
  if (blocks > 0x7FFFFFFF || n_slots < 1) return hipErrorInvalidValue;
  const dim3 grid(static_cast<unsigned>(blocks), n_slots), block(256);
  if (pass == CONV_WGRAD)
    hipLaunchKernelGGL(conv_update_kernel<CONV_WGRAD>, grid, block, 0, s, a, master, master_slot, lr);
  else
    hipLaunchKernelGGL(conv_update_kernel<FC_WGRAD>, grid, block, 0, s, a, master, master_slot, lr);
  return hipGetLastError();
}

hipError_t launch_avgpool(const float* act, int64_t act_slot, float* pooled, int64_t pooled_slot,
                          int B, int HW, int C, int n_slots, hipStream_t s) {
  const int64_t blocks = (static_cast<int64_t>(B) * C + 255) / 256;
  if (blocks > 0x7FFFFFFF || n_slots < 1) return hipErrorInvalidValue;
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

}  // namespace oscars
