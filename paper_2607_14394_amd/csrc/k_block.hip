// Point-wise linear layers over the points of a (B, C, V) tensor:
//
//   block epilogue (Sec. V "Block Structure", Algorithm 1 first and last
//   step), in place on the spectral output y:
//     y[b,o,n] <- GELU( sum_i w[o,i] x[b,i,n] + y[b,o,n] ),   GELU(v) = v Phi(v);
//   lift P and projection Q of the FNO (Sec. II), into a separate y:
//     y[b,o,n]  = act( sum_i w[o,i] x[b,i,n] + bias[o] ),   act = identity or GELU.
//
// Per point this is a (C_out x C_in) matrix-vector product, about
// 2 C_in C_out / (4 (C_in + 2 C_out)) flop per byte (2.7 at C = 16): bound by
// HBM traffic on x and y, so it runs on the VALU.  Each thread owns four
// consecutive points of one batch entry (16-byte accesses), reads their C_in
// input channels once per chunk of output channels (C_out rounded up to a
// multiple of 4 when that is at most 16, else chunks of 12 or 16), and reads
// w (and the bias) from LDS (the same entry for every lane).  GELU is the
// branch-free Abramowitz & Stegun 7.1.26 form of gelu_as.h (the library
// erff took about three times as many vector instructions).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "dtst_internal.h"

namespace dtst {
namespace {


#include "gelu_as.h"

// ADDY: the accumulators start from y (block epilogue), else from the bias
// (zero without one).  ACT: 1 applies GELU, 0 none.  OC: output channels per
// pass over the input channels (the launcher picks C_out rounded up to a
// multiple of 4 when that is at most 16, else 12 or 16).
template <int VEC, int ADDY, int ACT, int OC>
__global__ void __launch_bounds__(256)
pointwise_kernel(const float* __restrict__ x, const float* __restrict__ w, const float* __restrict__ bias,
                 float* __restrict__ y, int64_t V, int64_t total, int ci, int co) {
  // VEC: 4 points per thread (V % 4 == 0, 16-byte accesses), else 1.
  constexpr int P = VEC ? 4 : 1;
  const int64_t VP = V / P;
  // w (and the bias) in LDS: every lane reads the same entry (a broadcast),
  // which keeps them out of the scalar registers.
  extern __shared__ float sw[];
  float* sb = sw + co * ci;
  for (int e = threadIdx.x; e < co * ci; e += blockDim.x) sw[e] = w[e];
  if (!ADDY)
    for (int e = threadIdx.x; e < co; e += blockDim.x) sb[e] = bias ? bias[e] : 0.f;
  __syncthreads();
  for (int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; idx < total;
       idx += int64_t(gridDim.x) * blockDim.x) {
    const int64_t b = idx / VP, n = (idx - b * VP) * P;
    const float* xb = x + b * ci * V + n;
    float* yb = y + b * co * V + n;
    for (int o0 = 0; o0 < co; o0 += OC) {
      // the accumulators start from y (loaded before the x loop so that its
      // latency overlaps the reads of x) or from the bias
      float acc[OC][P];
#pragma unroll
      for (int oo = 0; oo < OC; ++oo) {
        const int o = o0 + oo < co ? o0 + oo : co - 1;
        const float* yp = yb + int64_t(o) * V;
        if constexpr (!ADDY) {
#pragma unroll
          for (int p = 0; p < P; ++p) acc[oo][p] = sb[o];
        } else if constexpr (VEC) {
          const float4 v = *reinterpret_cast<const float4*>(yp);
          acc[oo][0] = v.x;
          acc[oo][1] = v.y;
          acc[oo][2] = v.z;
          acc[oo][3] = v.w;
        } else {
          acc[oo][0] = *yp;
        }
      }
#pragma unroll 4
      for (int i = 0; i < ci; ++i) {
        float xv[P];
        if constexpr (VEC) {
          const float4 v = *reinterpret_cast<const float4*>(xb + int64_t(i) * V);
          xv[0] = v.x;
          xv[1] = v.y;
          xv[2] = v.z;
          xv[3] = v.w;
        } else {
          xv[0] = xb[int64_t(i) * V];
        }
#pragma unroll
        for (int oo = 0; oo < OC; ++oo) {
          const int o = o0 + oo < co ? o0 + oo : co - 1;
          const float wv = sw[o * ci + i];
#pragma unroll
          for (int p = 0; p < P; ++p) acc[oo][p] += wv * xv[p];
        }
      }
#pragma unroll
      for (int oo = 0; oo < OC; ++oo) {
        if (o0 + oo >= co) continue;
        float* yp = yb + int64_t(o0 + oo) * V;
        float r[P];
#pragma unroll
        for (int p = 0; p < P; ++p) r[p] = ACT ? gelu_as(acc[oo][p]) : acc[oo][p];
        if constexpr (VEC) {
          *reinterpret_cast<float4*>(yp) = make_float4(r[0], r[1], r[2], r[3]);
        } else {
          *yp = r[0];
        }
      }
    }
  }
}


template <int ADDY, int ACT, int OC>
int launch_pw_oc(const float* x, const float* w, const float* bias, float* y, int64_t B, int64_t ci, int64_t co,
                 int64_t V, void* stream) {
  const bool vec = V % 4 == 0;
  const int64_t total = B * (vec ? V / 4 : V);
  const int64_t cap = int64_t(1) << 20;
  const int64_t blocks = std::min<int64_t>((total + 255) / 256, cap);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t lds = (size_t(ci) * co + (ADDY ? 0 : co)) * sizeof(float);
  const void* fn = vec ? reinterpret_cast<const void*>(pointwise_kernel<1, ADDY, ACT, OC>)
                       : reinterpret_cast<const void*>(pointwise_kernel<0, ADDY, ACT, OC>);
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
  }
  if (vec)
    hipLaunchKernelGGL((pointwise_kernel<1, ADDY, ACT, OC>), dim3(static_cast<unsigned>(blocks)), dim3(256), lds, s,
                       x, w, bias, y, V, total, static_cast<int>(ci), static_cast<int>(co));
  else
    hipLaunchKernelGGL((pointwise_kernel<0, ADDY, ACT, OC>), dim3(static_cast<unsigned>(blocks)), dim3(256), lds, s,
                       x, w, bias, y, V, total, static_cast<int>(ci), static_cast<int>(co));
  return hipGetLastError();
}

template <int ADDY, int ACT>
int launch_pw(const float* x, const float* w, const float* bias, float* y, int64_t B, int64_t ci, int64_t co,
              int64_t V, void* stream) {
  if (B <= 0 || V <= 0) return hipSuccess;
  // C_out <= 16: one pass of C_out rounded up to a multiple of 4 (no wasted
  // products).  Wider layers take passes of 12 or 16, whichever computes
  // fewer unused outputs (a single wider pass held more registers and fewer
  // waves, and measured slower at C_out = 20).
  const int64_t waste12 = (co + 11) / 12 * 12 - co, waste16 = (co + 15) / 16 * 16 - co;
  const int pick = co <= 16 ? int((co + 3) / 4) : (waste12 < waste16 ? 3 : 4);
  switch (pick) {
    case 1: return launch_pw_oc<ADDY, ACT, 4>(x, w, bias, y, B, ci, co, V, stream);
    case 2: return launch_pw_oc<ADDY, ACT, 8>(x, w, bias, y, B, ci, co, V, stream);
    case 3: return launch_pw_oc<ADDY, ACT, 12>(x, w, bias, y, B, ci, co, V, stream);
    case 4: return launch_pw_oc<ADDY, ACT, 16>(x, w, bias, y, B, ci, co, V, stream);
    default: return launch_pw_oc<ADDY, ACT, 32>(x, w, bias, y, B, ci, co, V, stream);
  }
}

}  // namespace

int launch_block_epilogue(const float* x, const float* w, float* y, int64_t B, int64_t ci, int64_t co, int64_t V,
                          void* stream) {
  return launch_pw<1, 1>(x, w, nullptr, y, B, ci, co, V, stream);
}

int launch_pointwise(const float* x, const float* w, const float* bias, float* y, int64_t B, int64_t ci, int64_t co,
                     int64_t V, int act, void* stream) {
  return act ? launch_pw<0, 1>(x, w, bias, y, B, ci, co, V, stream)
             : launch_pw<0, 0>(x, w, bias, y, B, ci, co, V, stream);
}

}  // namespace dtst
