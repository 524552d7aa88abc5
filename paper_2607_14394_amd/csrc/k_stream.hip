// Streaming t+z kernels of the DTST library (gfx950, fp32 MFMA 16x16x4).
//
// Forward (Sec. IV-B Eq. dtst_decompose, first two of the per-dimension
// contractions of Sec. V-B, in the paper's order t then z): every wave takes
// one (N_z x N_t) row of the real shard, contracts t against the half-spectrum
// basis B_t and then z against B_z, and writes the (K_z x K_t) complex
// result.  The shard is read exactly once, with 16-byte loads; the row never
// leaves registers between the two contractions.
//
// Inverse (Sec. V-A Eq. dtst_inverse, last two expansions of the reverse
// order): every wave expands one (K_z x K_t) complex row over z and then
// over t, applying Re and the half-spectrum weights folded into the t
// basis, and writes the real (N_z x N_t) row.
//
// MFMA 16x16x4 fp32 lane layout (lane l, m = l & 15, g = l >> 4):
//   A operand: A[m][g], B operand: B[g][m], accumulator register i: C[4g+i][m].
// The K index seen by an instruction may be any permutation of the
// contraction index as long as A and B agree; the images built on the host
// use that freedom so that accumulators of one MFMA feed the next one
// without any data movement.
#include <hip/hip_runtime.h>

#include "dtst_internal.h"

namespace dtst {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4f mfma(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

struct StreamArgs {
  int64_t rows;
  int nt, nz, kt, kz, zh, zt, vec;
};

// ---------------------------------------------------------------------------
// Forward: x (rows x N_z x N_t) fp32 -> out (rows x K_z x K_t) complex.
// ---------------------------------------------------------------------------
template <int CT, int TH, int MT, int NCLS>
__global__ void __launch_bounds__(256)
fwd_tz_kernel(const float* __restrict__ x, float2* __restrict__ out,
              const float* __restrict__ timg, const float4* __restrict__ zimg, StreamArgs a) {
  extern __shared__ float4 lds[];
  const int nimg = NCLS * a.zt * MT * 64;
  for (int i = threadIdx.x; i < nimg; i += blockDim.x) lds[i] = zimg[i];
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  constexpr int KTP = 8 * CT;

  // B operand of the t contraction, step s = 4h + j covers t = 16h + 4g + j.
  float bt[TH * 4][CT];
#pragma unroll
  for (int s = 0; s < TH * 4; ++s)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) bt[s][ct] = timg[(s * CT + ct) * 64 + lane];

  const int wpb = blockDim.x >> 6;
  const int64_t wstride = int64_t(gridDim.x) * wpb;
  const int64_t row_len = int64_t(a.nz) * a.nt;

  for (int64_t r = int64_t(blockIdx.x) * wpb + (threadIdx.x >> 6); r < a.rows; r += wstride) {
    const float* xr = x + r * row_len;
    v4f P[NCLS][MT][CT];
#pragma unroll
    for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) P[cl][mt][ct] = v4f{0.f, 0.f, 0.f, 0.f};

    for (int zt = 0; zt < a.zt; ++zt) {
      const int zl = zt * 16 + m;
      const bool zok = zl < a.zh;
      // Contract t for z = zl (and z = zl + N_z/2 when folded).
      v4f V[NCLS][CT];
#pragma unroll
      for (int hf = 0; hf < NCLS; ++hf) {
        const float* src = xr + int64_t(zl + hf * a.zh) * a.nt;
        float xv[TH][4];
        if (a.vec) {
#pragma unroll
          for (int h = 0; h < TH; ++h) {
            const int t0 = 16 * h + 4 * g;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (zok && t0 < a.nt) v = *reinterpret_cast<const float4*>(src + t0);
            xv[h][0] = v.x; xv[h][1] = v.y; xv[h][2] = v.z; xv[h][3] = v.w;
          }
        } else {
#pragma unroll
          for (int h = 0; h < TH; ++h)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int t = 16 * h + 4 * g + j;
              xv[h][j] = (zok && t < a.nt) ? src[t] : 0.f;
            }
        }
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
          v4f acc = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int h = 0; h < TH; ++h)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc = mfma(xv[h][j], bt[h * 4 + j][ct], acc);
          V[hf][ct] = acc;
        }
      }
      if (NCLS == 2) {
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
          const v4f s = V[0][ct] + V[1][ct];
          const v4f d = V[0][ct] - V[1][ct];
          V[0][ct] = s;
          V[NCLS - 1][ct] = d;
        }
      }
      // Contract z: accumulator register i of V is the B operand of the
      // step whose K index is z = 16zt + 4g + i.
#pragma unroll
      for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const float4 A = lds[((cl * a.zt + zt) * MT + mt) * 64 + lane];
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) {
            v4f p = P[cl][mt][ct];
            p = mfma(A.x, V[cl][ct][0], p);
            p = mfma(A.y, V[cl][ct][1], p);
            p = mfma(A.z, V[cl][ct][2], p);
            p = mfma(A.w, V[cl][ct][3], p);
            P[cl][mt][ct] = p;
          }
        }
    }

    // Combine the real-stacked products into complex coefficients:
    // (Re B) V and (Im B) V sit in row tiles mt and mt + MT/2 of the same lane;
    // the Re / Im columns of k_t sit 8 lanes apart (CT = 1) or in the two
    // column tiles (CT = 2).
    float2* orow = out + r * int64_t(a.kz) * a.kt;
#pragma unroll
    for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
      for (int mr = 0; mr < MT / 2; ++mr)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int s = 16 * mr + 4 * g + i;
          const int p = s * NCLS + cl;
          if (CT == 1) {
            const float q = P[cl][mr][0][i];
            const float u = P[cl][mr + MT / 2][0][i];
            const float qs = __shfl_xor(q, 8);
            const float us = __shfl_xor(u, 8);
            if (m < KTP && m < a.kt && p < a.kz) orow[p * a.kt + m] = make_float2(q - us, qs + u);
          } else {
            const float rr = P[cl][mr][0][i], ri = P[cl][mr][CT - 1][i];
            const float ir = P[cl][mr + MT / 2][0][i], ii = P[cl][mr + MT / 2][CT - 1][i];
            if (m < a.kt && p < a.kz) orow[p * a.kt + m] = make_float2(rr - ii, ri + ir);
          }
        }
  }
}

// ---------------------------------------------------------------------------
// Inverse: in (rows x K_z x K_t) complex -> y (rows x N_z x N_t) fp32.
// ---------------------------------------------------------------------------
template <int CT, int TH, int MT, int NCLS>
__global__ void __launch_bounds__(256)
inv_zt_kernel(const float2* __restrict__ in, float* __restrict__ y,
              const float* __restrict__ timg, const float4* __restrict__ zimg, StreamArgs a) {
  extern __shared__ float4 lds[];
  const int nimg = NCLS * a.zt * MT * 64;
  for (int i = threadIdx.x; i < nimg; i += blockDim.x) lds[i] = zimg[i];
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  constexpr int KTP = 8 * CT;

  // A operand of the t expansion: rows t = 16mt + m, K index c = 16ct + 4g + i.
  float ta[TH][CT][4];
#pragma unroll
  for (int mt = 0; mt < TH; ++mt)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int i = 0; i < 4; ++i) ta[mt][ct][i] = timg[((mt * CT + ct) * 4 + i) * 64 + lane];

  const int wpb = blockDim.x >> 6;
  const int64_t wstride = int64_t(gridDim.x) * wpb;
  const int64_t row_len = int64_t(a.nz) * a.nt;

  for (int64_t r = int64_t(blockIdx.x) * wpb + (threadIdx.x >> 6); r < a.rows; r += wstride) {
    const float2* urow = in + r * int64_t(a.kz) * a.kt;
    // A operand of the z expansion (rows c, K index kz' = 16q + 4g + i):
    // kz' < KCP pairs with Re C_z, kz' >= KCP with Im C_z.
    float A[NCLS][CT][MT][4];
#pragma unroll
    for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int qh = 0; qh < MT / 2; ++qh)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int s = 16 * qh + 4 * g + i;
            const int p = s * NCLS + cl;
            const int c = 16 * ct + m;
            const bool is_re = c < KTP;
            const int kt = is_re ? c : c - KTP;
            float2 u = make_float2(0.f, 0.f);
            if (p < a.kz && kt < a.kt) u = urow[p * a.kt + kt];
            A[cl][ct][qh][i] = is_re ? u.x : u.y;
            A[cl][ct][qh + MT / 2][i] = is_re ? -u.y : u.x;
          }

    float* yrow = y + r * row_len;
    for (int zt = 0; zt < a.zt; ++zt) {
      v4f W[NCLS][CT];
#pragma unroll
      for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
          v4f acc = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int q = 0; q < MT; ++q) {
            const float4 B = lds[((cl * a.zt + zt) * MT + q) * 64 + lane];
            acc = mfma(A[cl][ct][q][0], B.x, acc);
            acc = mfma(A[cl][ct][q][1], B.y, acc);
            acc = mfma(A[cl][ct][q][2], B.z, acc);
            acc = mfma(A[cl][ct][q][3], B.w, acc);
          }
          W[cl][ct] = acc;
        }
      if (NCLS == 2) {
        // even modes + odd modes at z, even - odd at z + N_z/2
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
          const v4f s = W[0][ct] + W[NCLS - 1][ct];
          const v4f d = W[0][ct] - W[NCLS - 1][ct];
          W[0][ct] = s;
          W[NCLS - 1][ct] = d;
        }
      }
      const int zl = zt * 16 + m;
      const bool zok = zl < a.zh;
#pragma unroll
      for (int hf = 0; hf < NCLS; ++hf) {
        float* dst = yrow + int64_t(zl + hf * a.zh) * a.nt;
#pragma unroll
        for (int mt = 0; mt < TH; ++mt) {
          v4f Y = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) {
            Y = mfma(ta[mt][ct][0], W[hf][ct][0], Y);
            Y = mfma(ta[mt][ct][1], W[hf][ct][1], Y);
            Y = mfma(ta[mt][ct][2], W[hf][ct][2], Y);
            Y = mfma(ta[mt][ct][3], W[hf][ct][3], Y);
          }
          const int t0 = 16 * mt + 4 * g;
          if (a.vec) {
            if (zok && t0 < a.nt) *reinterpret_cast<float4*>(dst + t0) = make_float4(Y[0], Y[1], Y[2], Y[3]);
          } else if (zok) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (t0 + i < a.nt) dst[t0 + i] = Y[i];
          }
        }
      }
    }
  }
}

typedef void (*fwd_fn)(const float*, float2*, const float*, const float4*, StreamArgs);
typedef void (*inv_fn)(const float2*, float*, const float*, const float4*, StreamArgs);

template <int CT, int TH, int MT>
void pick2(int ncls, fwd_fn* f, inv_fn* v) {
  if (ncls == 2) {
    *f = fwd_tz_kernel<CT, TH, MT, 2>;
    *v = inv_zt_kernel<CT, TH, MT, 2>;
  } else {
    *f = fwd_tz_kernel<CT, TH, MT, 1>;
    *v = inv_zt_kernel<CT, TH, MT, 1>;
  }
}

template <int CT, int TH>
void pick1(int mt, int ncls, fwd_fn* f, inv_fn* v) {
  if (mt == 2) pick2<CT, TH, 2>(ncls, f, v);
  else if (mt == 4) pick2<CT, TH, 4>(ncls, f, v);
  else pick2<CT, TH, 8>(ncls, f, v);
}

template <int CT>
void pick0(int th, int mt, int ncls, fwd_fn* f, inv_fn* v) {
  if (th == 1) pick1<CT, 1>(mt, ncls, f, v);
  else if (th == 2) pick1<CT, 2>(mt, ncls, f, v);
  else pick1<CT, 4>(mt, ncls, f, v);
}

void pick(const StreamCfg& c, fwd_fn* f, inv_fn* v) {
  if (c.ct == 1) pick0<1>(c.th, c.mt, c.ncls, f, v);
  else pick0<2>(c.th, c.mt, c.ncls, f, v);
}

StreamArgs args_of(const StreamCfg& c, int64_t rows) {
  StreamArgs a;
  a.rows = rows;
  a.nt = c.nt;
  a.nz = c.nz;
  a.kt = c.kt;
  a.kz = c.kz;
  a.zh = c.zh;
  a.zt = c.zt;
  a.vec = c.vec;
  return a;
}

int resident_grid(const void* fn, size_t lds) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 256, lds) != hipSuccess) return 0;
  return cus * (per_cu > 0 ? per_cu : 1);
}

int grid_for(int resident, int64_t rows) {
  const int64_t want = (rows + 3) / 4;
  return static_cast<int>(want < resident ? want : resident);
}

}  // namespace

int prepare_stream(StreamCfg* c) {
  fwd_fn f;
  inv_fn v;
  pick(*c, &f, &v);
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(f),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(c->lds_bytes));
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(v), hipFuncAttributeMaxDynamicSharedMemorySize,
                          int(c->lds_bytes));
  if (e != hipSuccess) return e;
  c->grid_fwd = resident_grid(reinterpret_cast<const void*>(f), c->lds_bytes);
  c->grid_inv = resident_grid(reinterpret_cast<const void*>(v), c->lds_bytes);
  if (c->grid_fwd <= 0 || c->grid_inv <= 0) return hipErrorInvalidConfiguration;
  return hipSuccess;
}

int launch_fwd_tz(const StreamCfg& c, const float* x, void* out, int64_t rows, const float* timg,
                  const float* zimg, void* stream) {
  if (rows <= 0) return hipSuccess;
  fwd_fn f;
  inv_fn v;
  pick(c, &f, &v);
  hipLaunchKernelGGL(f, dim3(grid_for(c.grid_fwd, rows)), dim3(256), c.lds_bytes, static_cast<hipStream_t>(stream),
                     x, static_cast<float2*>(out), timg, reinterpret_cast<const float4*>(zimg), args_of(c, rows));
  return hipGetLastError();
}

int launch_inv_zt(const StreamCfg& c, const void* in, float* y, int64_t rows, const float* timg,
                  const float* zimg, void* stream) {
  if (rows <= 0) return hipSuccess;
  fwd_fn f;
  inv_fn v;
  pick(c, &f, &v);
  hipLaunchKernelGGL(v, dim3(grid_for(c.grid_inv, rows)), dim3(256), c.lds_bytes, static_cast<hipStream_t>(stream),
                     static_cast<const float2*>(in), y, timg, reinterpret_cast<const float4*>(zimg),
                     args_of(c, rows));
  return hipGetLastError();
}

}  // namespace dtst
