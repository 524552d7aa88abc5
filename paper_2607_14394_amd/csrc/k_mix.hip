// Mode-wise channel mix and its gradients (Sec. V-A Eq. partitioned_conv,
// Sec. V-C), on a flattened mode range [m0, m1):
//
//   mix      yhat[b,o,m] = sum_i xhat[b,i,m] w[m-m0,i,o]
//   mix_h    g_x[b,i,m]  = sum_o g_y[b,o,m] conj(w[m-m0,i,o])     (data gradient)
//   wgrad    g_w[m-m0,i,o] (+)= sum_b conj(xhat[b,i,m]) g_y[b,o,m]
//
// With B <= 2 the arithmetic intensity is about 1-2 flop/byte, so all three
// are bound by HBM traffic on w / g_w (M C_in C_out complex values).  Each
// workgroup owns a block of consecutive modes: the spectra of those modes
// (stride M between channels) are staged through LDS so that every global
// access is coalesced, and w / g_w are streamed in their natural
// (m, i, o) order.
#include <hip/hip_runtime.h>

#include "dtst_internal.h"

namespace dtst {
namespace {

struct MixArgs {
  int64_t M, m0, count;  // count = m1 - m0
  int64_t nblk;           // number of mode blocks
  int B, ci, co, mpb;     // mpb = modes per block
  int acc;
};

__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
  return make_float2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
// conj(a) * b
__device__ __forceinline__ float2 cjmul(float2 a, float2 b) {
  return make_float2(a.x * b.x + a.y * b.y, a.x * b.y - a.y * b.x);
}

constexpr int BCH = 4;  // batch entries accumulated per pass

// Stage spec[b][c][mbase .. mbase+nm) (channels C) into LDS as [b][c][mm].
__device__ __forceinline__ void stage(float2* dst, const float2* __restrict__ spec, int B, int C, int64_t M,
                                      int64_t mbase, int nm, int mpb) {
  const int n = B * C * nm;
  for (int e = threadIdx.x; e < n; e += blockDim.x) {
    const int mm = e % nm;
    const int bc = e / nm;
    dst[bc * mpb + mm] = spec[int64_t(bc) * M + mbase + mm];
  }
}

__device__ __forceinline__ void unstage(float2* __restrict__ spec, const float2* src, int B, int C, int64_t M,
                                        int64_t mbase, int nm, int mpb) {
  const int n = B * C * nm;
  for (int e = threadIdx.x; e < n; e += blockDim.x) {
    const int mm = e % nm;
    const int bc = e / nm;
    spec[int64_t(bc) * M + mbase + mm] = src[bc * mpb + mm];
  }
}

__global__ void __launch_bounds__(256)
mix_kernel(const float2* __restrict__ x, const float2* __restrict__ w, float2* __restrict__ y, MixArgs a) {
  extern __shared__ float2 sm[];
  float2* sx = sm;                          // [B][ci][mpb]
  float2* sy = sm + a.B * a.ci * a.mpb;     // [B][co][mpb]
  for (int64_t blk = blockIdx.x; blk < a.nblk; blk += gridDim.x) {
  const int64_t lm0 = blk * a.mpb;  // local mode index in [0, count)
  const int nm = static_cast<int>(min(int64_t(a.mpb), a.count - lm0));
  const int64_t mbase = a.m0 + lm0;
  stage(sx, x, a.B, a.ci, a.M, mbase, nm, a.mpb);
  __syncthreads();
  for (int e = threadIdx.x; e < nm * a.co; e += blockDim.x) {
    const int o = e % a.co;
    const int mm = e / a.co;
    const float2* wp = w + (lm0 + mm) * int64_t(a.ci) * a.co + o;
    for (int b0 = 0; b0 < a.B; b0 += BCH) {
      float2 acc[BCH];
#pragma unroll
      for (int q = 0; q < BCH; ++q) acc[q] = make_float2(0.f, 0.f);
      for (int i = 0; i < a.ci; ++i) {
        const float2 wv = wp[int64_t(i) * a.co];
#pragma unroll
        for (int q = 0; q < BCH; ++q) {
          if (b0 + q < a.B) {
            const float2 xv = sx[((b0 + q) * a.ci + i) * a.mpb + mm];
            const float2 p = cmul(xv, wv);
            acc[q].x += p.x;
            acc[q].y += p.y;
          }
        }
      }
#pragma unroll
      for (int q = 0; q < BCH; ++q)
        if (b0 + q < a.B) sy[((b0 + q) * a.co + o) * a.mpb + mm] = acc[q];
    }
  }
  __syncthreads();
  unstage(y, sy, a.B, a.co, a.M, mbase, nm, a.mpb);
  __syncthreads();
  }
}

// Data gradient: the w block of the workgroup's modes is staged in LDS
// (row stride 2*co + 2 floats, so lanes reading consecutive rows i hit
// different banks) and each thread owns one (mode, i) pair.
__global__ void __launch_bounds__(256)
mix_h_kernel(const float2* __restrict__ gy, const float2* __restrict__ w, float2* __restrict__ gx, MixArgs a) {
  extern __shared__ float2 sm[];
  const int wrow = a.co + 1;                           // float2 stride of one (mode, i) row
  float2* sw = sm;                                     // [mpb][ci][wrow]
  float2* sg = sw + a.mpb * a.ci * wrow;               // [B][co][mpb]
  float2* sx = sg + a.B * a.co * a.mpb;                // [B][ci][mpb]
  for (int64_t blk = blockIdx.x; blk < a.nblk; blk += gridDim.x) {
  const int64_t lm0 = blk * a.mpb;
  const int nm = static_cast<int>(min(int64_t(a.mpb), a.count - lm0));
  const int64_t mbase = a.m0 + lm0;
  stage(sg, gy, a.B, a.co, a.M, mbase, nm, a.mpb);
  const int nw = nm * a.ci * a.co;
  const float2* wb = w + lm0 * int64_t(a.ci) * a.co;
  for (int e = threadIdx.x; e < nw; e += blockDim.x) {
    const int o = e % a.co;
    const int mi = e / a.co;  // mm * ci + i
    sw[mi * wrow + o] = wb[e];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < nm * a.ci; e += blockDim.x) {
    const int i = e % a.ci;
    const int mm = e / a.ci;
    const float2* wr = sw + (mm * a.ci + i) * wrow;
    for (int b0 = 0; b0 < a.B; b0 += BCH) {
      float2 acc[BCH];
#pragma unroll
      for (int q = 0; q < BCH; ++q) acc[q] = make_float2(0.f, 0.f);
      for (int o = 0; o < a.co; ++o) {
        const float2 wv = wr[o];
#pragma unroll
        for (int q = 0; q < BCH; ++q) {
          if (b0 + q < a.B) {
            const float2 gv = sg[((b0 + q) * a.co + o) * a.mpb + mm];
            const float2 p = cjmul(wv, gv);
            acc[q].x += p.x;
            acc[q].y += p.y;
          }
        }
      }
#pragma unroll
      for (int q = 0; q < BCH; ++q)
        if (b0 + q < a.B) sx[((b0 + q) * a.ci + i) * a.mpb + mm] = acc[q];
    }
  }
  __syncthreads();
  unstage(gx, sx, a.B, a.ci, a.M, mbase, nm, a.mpb);
  __syncthreads();
  }
}

__global__ void __launch_bounds__(256)
wgrad_kernel(const float2* __restrict__ x, const float2* __restrict__ gy, float2* __restrict__ gw, MixArgs a) {
  extern __shared__ float2 sm[];
  float2* sx = sm;                       // [B][ci][mpb]
  float2* sg = sm + a.B * a.ci * a.mpb;  // [B][co][mpb]
  for (int64_t blk = blockIdx.x; blk < a.nblk; blk += gridDim.x) {
  const int64_t lm0 = blk * a.mpb;
  const int nm = static_cast<int>(min(int64_t(a.mpb), a.count - lm0));
  const int64_t mbase = a.m0 + lm0;
  stage(sx, x, a.B, a.ci, a.M, mbase, nm, a.mpb);
  stage(sg, gy, a.B, a.co, a.M, mbase, nm, a.mpb);
  __syncthreads();
  for (int e = threadIdx.x; e < nm * a.co; e += blockDim.x) {
    const int o = e % a.co;
    const int mm = e / a.co;
    float2* gp = gw + (lm0 + mm) * int64_t(a.ci) * a.co + o;
    for (int i = 0; i < a.ci; ++i) {
      float2 acc = make_float2(0.f, 0.f);
      for (int b = 0; b < a.B; ++b) {
        const float2 p = cjmul(sx[(b * a.ci + i) * a.mpb + mm], sg[(b * a.co + o) * a.mpb + mm]);
        acc.x += p.x;
        acc.y += p.y;
      }
      float2* dst = gp + int64_t(i) * a.co;
      if (a.acc) {
        const float2 old = *dst;
        acc.x += old.x;
        acc.y += old.y;
      }
      *dst = acc;
    }
  }
  __syncthreads();
  }
}

// Modes per block: enough (mode, channel) work items for 256 threads, capped
// so the staged tiles fit in 64 KiB of LDS.
int modes_per_block(int per_mode_items, size_t per_mode_lds) {
  int mpb = 256 / (per_mode_items > 0 ? per_mode_items : 1);
  if (mpb < 1) mpb = 1;
  if (mpb > 64) mpb = 64;
  while (mpb > 1 && size_t(mpb) * per_mode_lds > 64 * 1024) --mpb;
  return mpb;
}

MixArgs make_args(int64_t B, int64_t ci, int64_t co, int64_t M, int64_t m0, int64_t m1, int mpb, int acc) {
  MixArgs a;
  a.M = M;
  a.m0 = m0;
  a.count = m1 - m0;
  a.B = static_cast<int>(B);
  a.ci = static_cast<int>(ci);
  a.co = static_cast<int>(co);
  a.mpb = mpb;
  a.acc = acc;
  a.nblk = (a.count + mpb - 1) / mpb;
  return a;
}

}  // namespace

// Largest LDS a mix launch may need; the host checks this before launching.
size_t mix_lds_bytes(int op, int64_t B, int64_t ci, int64_t co) {
  const size_t c8 = sizeof(float2);
  if (op == 1) return c8 * (size_t(ci) * (co + 1) + size_t(B) * (ci + co));
  return c8 * size_t(B) * (ci + co);
}

int launch_mix(const void* xhat, const void* w, void* yhat, int64_t B, int64_t ci, int64_t co, int64_t M,
               int64_t m0, int64_t m1, void* stream) {
  if (B <= 0 || m1 <= m0) return hipSuccess;
  const size_t per_mode = mix_lds_bytes(0, B, ci, co);
  const int mpb = modes_per_block(static_cast<int>(co), per_mode);
  const MixArgs a = make_args(B, ci, co, M, m0, m1, mpb, 0);
  const int64_t blocks = a.nblk < (int64_t(1) << 22) ? a.nblk : (int64_t(1) << 22);
  if (per_mode * mpb > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(mix_kernel),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, int(per_mode * mpb));
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(mix_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), per_mode * mpb,
                     static_cast<hipStream_t>(stream), static_cast<const float2*>(xhat),
                     static_cast<const float2*>(w), static_cast<float2*>(yhat), a);
  return hipGetLastError();
}

int launch_mix_h(const void* gy, const void* w, void* gx, int64_t B, int64_t ci, int64_t co, int64_t M,
                 int64_t m0, int64_t m1, void* stream) {
  if (B <= 0 || m1 <= m0) return hipSuccess;
  const size_t per_mode = mix_lds_bytes(1, B, ci, co);
  const int mpb = modes_per_block(static_cast<int>(ci), per_mode);
  const MixArgs a = make_args(B, ci, co, M, m0, m1, mpb, 0);
  const int64_t blocks = a.nblk < (int64_t(1) << 22) ? a.nblk : (int64_t(1) << 22);
  if (per_mode * mpb > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(mix_h_kernel),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, int(per_mode * mpb));
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(mix_h_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), per_mode * mpb,
                     static_cast<hipStream_t>(stream), static_cast<const float2*>(gy),
                     static_cast<const float2*>(w), static_cast<float2*>(gx), a);
  return hipGetLastError();
}

int launch_wgrad(const void* xhat, const void* gy, void* gw, int64_t B, int64_t ci, int64_t co, int64_t M,
                 int64_t m0, int64_t m1, int accumulate, void* stream) {
  if (B <= 0 || m1 <= m0) return hipSuccess;
  const size_t per_mode = mix_lds_bytes(0, B, ci, co);
  const int mpb = modes_per_block(static_cast<int>(co), per_mode);
  const MixArgs a = make_args(B, ci, co, M, m0, m1, mpb, accumulate ? 1 : 0);
  const int64_t blocks = a.nblk < (int64_t(1) << 22) ? a.nblk : (int64_t(1) << 22);
  if (per_mode * mpb > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(wgrad_kernel),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, int(per_mode * mpb));
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(wgrad_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), per_mode * mpb,
                     static_cast<hipStream_t>(stream), static_cast<const float2*>(xhat),
                     static_cast<const float2*>(gy), static_cast<float2*>(gw), a);
  return hipGetLastError();
}

}  // namespace dtst
