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

__host__ __device__ inline Dims pass_dims(const ConvArgs& a, int pass) {
  switch (pass) {
    case CONV_FWD: return {static_cast<int64_t>(a.B) * a.Ho * a.Wo, a.Co, 9LL * a.C};
    case CONV_DGRAD: return {static_cast<int64_t>(a.B) * a.H * a.W, a.C, 9LL * a.Co};
    case CONV_WGRAD: return {a.Co, 9LL * a.C + 1, static_cast<int64_t>(a.B) * a.Ho * a.Wo};
    case FC_FWD: return {a.B, a.Co, a.C};
    case FC_DGRAD: return {a.B, a.C, a.Co};
    default: return {a.Co, static_cast<int64_t>(a.C) + 1, a.B};  // FC_WGRAD
  }
}

// Input tap k = (r 3 + s) C + c of output pixel `pix` = (b Ho + i) Wo + j:
// input[b][stride i + r - 1][stride j + s - 1][c], zero outside the image.
__device__ __forceinline__ float conv_tap(const ConvArgs& a, const float* in,
                                          const int32_t* rows, int64_t pix, int64_t k) {
  const int64_t hw = static_cast<int64_t>(a.Ho) * a.Wo;
  const int b = static_cast<int>(pix / hw), p = static_cast<int>(pix % hw);
  const int i = p / a.Wo, j = p % a.Wo;
  const int rs = static_cast<int>(k / a.C), c = static_cast<int>(k % a.C);
  const int hi = a.stride * i + rs / 3 - 1, wi = a.stride * j + rs % 3 - 1;
  if (hi < 0 || hi >= a.H || wi < 0 || wi >= a.W) return 0.0f;
  const float* img = rows ? in + static_cast<int64_t>(rows[b]) * a.in_ld
                          : in + static_cast<int64_t>(b) * a.H * a.W * a.C;
  return img[(static_cast<int64_t>(hi) * a.W + wi) * a.C + c];
}

// Output-gradient tap k = (r 3 + s) Cout + o of input pixel q = (b H + hi) W + wi:
// dZ[b][i][j][o] where stride i + r - 1 = hi and stride j + s - 1 = wi, else 0.
__device__ __forceinline__ float dgrad_tap(const ConvArgs& a, const float* dz, int64_t q,
                                           int64_t k) {
  const int64_t hw = static_cast<int64_t>(a.H) * a.W;
  const int b = static_cast<int>(q / hw), p = static_cast<int>(q % hw);
  const int hi = p / a.W, wi = p % a.W;
  const int rs = static_cast<int>(k / a.Co), o = static_cast<int>(k % a.Co);
  const int ti = hi + 1 - rs / 3, tj = wi + 1 - rs % 3;
  if (ti < 0 || tj < 0 || ti % a.stride != 0 || tj % a.stride != 0) return 0.0f;
  const int i = ti / a.stride, j = tj / a.stride;
  if (i >= a.Ho || j >= a.Wo) return 0.0f;
  return dz[((static_cast<int64_t>(b) * a.Ho + i) * a.Wo + j) * a.Co + o];
}

template <int PASS>
__global__ __launch_bounds__(256) void conv_gemm_kernel(ConvArgs a) {
  constexpr bool WG = PASS == CONV_WGRAD || PASS == FC_WGRAD;
  __shared__ float As[2][CK][CLD];
  __shared__ float Bs[2][CK][CLD];
  const Dims d = pass_dims(a, PASS);
  const int z = blockIdx.y;
  const int rep = a.order[z];
  const int64_t gm = (d.M + CT - 1) / CT, gn = (d.N + CT - 1) / CT;
  int64_t tile = blockIdx.x;
  int split = 0;
  if constexpr (WG) {
    split = static_cast<int>(tile / (gm * gn));
    tile %= gm * gn;
  }
  const int64_t m0 = tile / gn * CT, n0 = tile % gn * CT;
  const int64_t kbeg = WG ? split * a.k_per_split : 0;
  const int64_t kend = WG ? (d.K < kbeg + a.k_per_split ? d.K : kbeg + a.k_per_split) : d.K;

  const float* in = a.in ? a.in + z * a.in_slot : nullptr;
  const int32_t* rows = a.gather ? a.gather + z * a.gather_slot : nullptr;
  const float* dz = a.dout ? a.dout + z * a.dout_slot : nullptr;
  const float* par = a.master_in + static_cast<int64_t>(rep) * a.master_in_slot;
  const float* Wt = par + a.w_off;

  auto A = [&](int64_t m, int64_t k) -> float {
    if constexpr (PASS == CONV_FWD) return conv_tap(a, in, rows, m, k);
    if constexpr (PASS == CONV_DGRAD) return dgrad_tap(a, dz, m, k);
    if constexpr (PASS == CONV_WGRAD) return dz[k * a.Co + m];
    if constexpr (PASS == FC_FWD) return in[m * a.C + k];
    if constexpr (PASS == FC_DGRAD) return dz[m * a.dout_ld + k];
    return dz[k * a.dout_ld + m];  // FC_WGRAD
  };
  auto Bv = [&](int64_t n, int64_t k) -> float {
    if constexpr (PASS == CONV_FWD) return Wt[n * 9 * a.C + k];
    if constexpr (PASS == CONV_DGRAD) return Wt[(k % a.Co) * 9 * a.C + (k / a.Co) * a.C + n];
    if constexpr (PASS == CONV_WGRAD) return n == 9LL * a.C ? 1.0f : conv_tap(a, in, rows, k, n);
    if constexpr (PASS == FC_FWD) return Wt[n * a.C + k];
    if constexpr (PASS == FC_DGRAD) return Wt[k * a.C + n];
    return n == a.C ? 1.0f : in[k * a.C + n];  // FC_WGRAD
  };

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, r = lane & 31, h = lane >> 5;
  // loader: thread t gathers rows m0 + t / 4 (A) and n0 + t / 4 (B), K
  // elements 4 (t % 4) .. 4 (t % 4) + 3 of the step
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  float ra[4], rb[4];
  auto gather = [&](int64_t k0) {
    const int64_t m = m0 + lr, n = n0 + lr;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t k = k0 + lk + e;
      ra[e] = (m < d.M && k < kend) ? A(m, k) : 0.0f;
      rb[e] = (n < d.N && k < kend) ? Bv(n, k) : 0.0f;
    }
  };
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
  const int64_t nk = (kend - kbeg + CK - 1) / CK;
  gather(kbeg);
  stash(0);
  __syncthreads();
  for (int64_t t = 0; t < nk; ++t) {
    const int buf = static_cast<int>(t & 1);
    if (t + 1 < nk) gather(kbeg + (t + 1) * CK);
    // MFMA u contracts k = 2u (lanes 0-31) and 2u + 1 (lanes 32-63)
#pragma unroll
    for (int u = 0; u < CK / 2; ++u)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(As[buf][2 * u + h][wm * 32 + r],
                                                 Bs[buf][2 * u + h][wn * 32 + r], acc, 0, 0, 0);
    if (t + 1 < nk) stash(buf ^ 1);
    __syncthreads();
  }

  // accumulator i of lane (r, h): row 8 (i / 4) + 4 h + i % 4, column r
  const int64_t col = n0 + wn * 32 + r;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int64_t row = m0 + wm * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
    if (row >= d.M || col >= d.N) continue;
    const float v = acc[i];
    if constexpr (PASS == CONV_FWD) {
      const float zv = v + par[a.b_off + col];
      a.out[z * a.out_slot + row * a.Co + col] = zv > 0.0f ? zv : 0.0f;
    } else if constexpr (PASS == FC_FWD) {
      a.out[z * a.out_slot + row * a.out_ld + col] = v + par[a.b_off + col];
    } else if constexpr (PASS == CONV_DGRAD) {
      const int64_t at = row * a.C + col;
      a.out[z * a.out_slot + at] = a.mask[z * a.mask_slot + at] > 0.0f ? v : 0.0f;
    } else if constexpr (PASS == FC_DGRAD) {
      a.out[z * a.out_slot + row * a.out_ld + col] = v;
    } else {
      a.part[z * a.part_slot + (split * d.M + row) * d.N + col] = v;
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
