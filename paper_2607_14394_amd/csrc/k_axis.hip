// Complex contraction along a middle axis (gfx950, fp32 MFMA 16x16x4):
//
//   out[b][k][n] (+)= sum_j basis[k][j] in[b][j][n]
//
// This is one per-dimension partial-DFT step of Sec. V-B: forward y
// (j = y, k = k_y), forward x with the shard-sum accumulate of Eq.
// (dtst_reduce) (j = x, k = k_x), and the inverse expansions over x and y
// with conj(B)^T (Sec. V-A Eq. dtst_inverse, reverse order).  The complex
// product is done as four real MFMA products with the basis split into
// (Re, Im, -Im) parts, so the epilogue is lane-local.
//
// Work split: a 256-thread workgroup owns one b, 64 consecutive n (16 per
// wave) and a block of up to KT*16 rows k.  Every lane streams in[b][j][n]
// for its n with 8-byte loads (16 lanes cover 128 contiguous bytes); the
// basis image is read with 16-byte loads that hit in L1/L2.
#include <hip/hip_runtime.h>

#include "dtst_internal.h"

namespace dtst {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4f mfma(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

struct AxisArgs {
  int64_t nb, total;
  int J, KO, NN, JQ, ktiles, kblocks, nblocks, acc;
};

// Blocks are dispatched round-robin over the 8 XCDs; give each XCD a
// contiguous range of logical tiles so the k blocks that re-read one input
// tile share an L2.
__device__ __forceinline__ int64_t xcd_logical(int64_t bid, int64_t grid) {
  const int64_t per = grid / 8;
  if (bid >= per * 8) return bid;
  return (bid % 8) * per + bid / 8;
}

template <int KT>
__global__ void __launch_bounds__(256)
axis_kernel(const float2* __restrict__ in, float2* __restrict__ out, const float4* __restrict__ img,
            AxisArgs a) {
  const int lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int wave = threadIdx.x >> 6;
  for (int64_t hw = blockIdx.x; hw < a.total; hw += gridDim.x) {
    const int64_t grid_round = (hw / gridDim.x == (a.total - 1) / gridDim.x)
                                   ? a.total - (hw / gridDim.x) * gridDim.x
                                   : int64_t(gridDim.x);
    const int64_t base = (hw / gridDim.x) * gridDim.x;
    const int64_t L = base + xcd_logical(hw - base, grid_round);
    const int nbk = static_cast<int>(L % a.nblocks);
    const int64_t rest = L / a.nblocks;
    const int kb = static_cast<int>(rest % a.kblocks);
    const int64_t b = rest / a.kblocks;

    const int n = nbk * 64 + wave * 16 + m;
    const bool nok = n < a.NN;
    const float2* inb = in + b * int64_t(a.J) * a.NN + n;

    v4f accr[KT], acci[KT];
#pragma unroll
    for (int kk = 0; kk < KT; ++kk) {
      accr[kk] = v4f{0.f, 0.f, 0.f, 0.f};
      acci[kk] = v4f{0.f, 0.f, 0.f, 0.f};
    }

    for (int q = 0; q < a.JQ; ++q) {
      float2 v[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = 16 * q + 4 * g + i;
        v[i] = (nok && j < a.J) ? inb[int64_t(j) * a.NN] : make_float2(0.f, 0.f);
      }
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) {
        const int kt = kb * KT + kk;
        if (kt < a.ktiles) {
          const float4* ip = img + (int64_t(kt) * a.JQ + q) * 3 * 64 + lane;
          const float4 br = ip[0], bi = ip[64], nbi = ip[128];
          v4f r = accr[kk], s = acci[kk];
          r = mfma(br.x, v[0].x, r); r = mfma(nbi.x, v[0].y, r);
          s = mfma(br.x, v[0].y, s); s = mfma(bi.x, v[0].x, s);
          r = mfma(br.y, v[1].x, r); r = mfma(nbi.y, v[1].y, r);
          s = mfma(br.y, v[1].y, s); s = mfma(bi.y, v[1].x, s);
          r = mfma(br.z, v[2].x, r); r = mfma(nbi.z, v[2].y, r);
          s = mfma(br.z, v[2].y, s); s = mfma(bi.z, v[2].x, s);
          r = mfma(br.w, v[3].x, r); r = mfma(nbi.w, v[3].y, r);
          s = mfma(br.w, v[3].y, s); s = mfma(bi.w, v[3].x, s);
          accr[kk] = r;
          acci[kk] = s;
        }
      }
    }

#pragma unroll
    for (int kk = 0; kk < KT; ++kk) {
      const int kt = kb * KT + kk;
      if (kt < a.ktiles && nok) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int k = 16 * kt + 4 * g + i;
          if (k < a.KO) {
            float2* o = out + (b * a.KO + k) * int64_t(a.NN) + n;
            float2 val = make_float2(accr[kk][i], acci[kk][i]);
            if (a.acc) {
              const float2 old = *o;
              val.x += old.x;
              val.y += old.y;
            }
            *o = val;
          }
        }
      }
    }
  }
}

}  // namespace

int launch_axis(const AxisCfg& c, int64_t nb, const void* in, void* out, const float* img, int accumulate,
                void* stream) {
  if (nb <= 0) return hipSuccess;
  AxisArgs a;
  a.nb = nb;
  a.J = c.J;
  a.KO = c.KO;
  a.NN = c.NN;
  a.JQ = c.JQ;
  a.ktiles = c.ktiles;
  a.acc = accumulate ? 1 : 0;
  a.nblocks = (c.NN + 63) / 64;
  int kt = c.ktiles <= 1 ? 1 : (c.ktiles <= 2 ? 2 : 4);
  a.kblocks = (c.ktiles + kt - 1) / kt;
  a.total = nb * a.kblocks * a.nblocks;
  const int64_t cap = int64_t(1) << 22;
  const int grid = static_cast<int>(a.total < cap ? a.total : cap);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const float2* pin = static_cast<const float2*>(in);
  float2* pout = static_cast<float2*>(out);
  const float4* pimg = reinterpret_cast<const float4*>(img);
  if (kt == 1) hipLaunchKernelGGL(axis_kernel<1>, dim3(grid), dim3(256), 0, s, pin, pout, pimg, a);
  else if (kt == 2) hipLaunchKernelGGL(axis_kernel<2>, dim3(grid), dim3(256), 0, s, pin, pout, pimg, a);
  else hipLaunchKernelGGL(axis_kernel<4>, dim3(grid), dim3(256), 0, s, pin, pout, pimg, a);
  return hipGetLastError();
}

}  // namespace dtst
