// Mode-wise channel mix and its gradients (Sec. V-A Eq. partitioned_conv,
// Sec. V-C), on a flattened mode range [m0, m1):
//
//   mix      yhat[b,o,m] = sum_i xhat[b,i,m] w[m-m0,i,o]
//   mix_h    g_x[b,i,m]  = sum_o g_y[b,o,m] conj(w[m-m0,i,o])     (data gradient)
//   wgrad    g_w[m-m0,i,o] (+)= sum_b conj(xhat[b,i,m]) g_y[b,o,m]
//
// With B <= 2 the arithmetic intensity is about 1-2 flop/byte, so all three
// are bound by HBM traffic on w / g_w (M C_in C_out complex values).
//
// Layout of the work: a "row group" of LPR lanes (the power of two >= C_out,
// at most 64) covers one row (m, i, 0..C_out) of w / g_w, lane l holding the
// columns o = l + LPR s (s < OPL), so every row is read or written with
// contiguous 8-byte accesses.  A 256-thread workgroup has 256 / LPR groups and
// handles that many consecutive modes at a time ("mode block"), one per
// group.  The spectra of a block (stride M between channels in HBM) are
// staged through LDS as [b][channel][mode + 1], which turns their strided
// reads into coalesced ones and gives each group its per-mode vectors.
//
// mix and mix_h (bound by the reads of w): one workgroup per mode block in
// an XCD-aware order; the first rows of w are loaded into registers before
// the staging barrier, so their HBM latency overlaps the staging.
// wgrad (bound by the writes of g_w): a grid of resident workgroups, each
// walking a contiguous run of mode blocks (its reads of the spectra advance
// through the same DRAM rows), fetching the next block's spectra into
// registers while the current block's rows are written, with the LDS area
// double-buffered so that one barrier per block separates writers and
// readers.
#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>

#include "dtst_internal.h"

namespace dtst {
namespace {

struct MixArgs {
  int64_t M, m0, count;  // count = m1 - m0
  int64_t nblk;           // number of mode blocks
  int B, ci, co;
  int lpr, mpb;           // lanes per row group, modes per block (= 256 / lpr)
  int acc;
};

typedef float v2f __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));

// Spectrum entries of one batch chunk processed together.
constexpr int BCH = 2;

// w rows held in registers per chunk (times OPL columns per lane).
template <int OPL>
struct Rows {
  static constexpr int value = OPL >= 8 ? 2 : 16 / OPL;
};

// Spectra of a block's modes in LDS: entry (b, c, mm) at
// [(b * C + c) * (MPB + 1) + mm].  They are read from spec[b][c][mbase + mm]
// (channel stride M), MPB consecutive modes per (b, c) row; each thread
// fetches its PRE entries into registers one block ahead and writes them to
// LDS when that block starts (entries beyond 256 * PRE are copied directly).
constexpr int PRE = 4;

template <int MPB>
__device__ __forceinline__ int sidx(int bc, int mm) {
  return bc * (MPB + 1) + mm;
}

// Direct staging of a block's spectra (no register prefetch).
template <int MPB>
__device__ __forceinline__ void stage(float2* dst, const float2* __restrict__ spec, int BC, int64_t M,
                                      int64_t mbase, int nm) {
  for (int e = threadIdx.x; e < BC * MPB; e += 256) {
    const int mm = e % MPB, bc = e / MPB;
    if (mm < nm) dst[sidx<MPB>(bc, mm)] = spec[int64_t(bc) * M + mbase + mm];
  }
}

template <int MPB>
__device__ __forceinline__ void fetch(float2 (&pre)[PRE], const float2* __restrict__ spec, int BC, int64_t M,
                                      int64_t mbase, int nm) {
#pragma unroll
  for (int j = 0; j < PRE; ++j) {
    const int e = threadIdx.x + 256 * j;
    const int mm = e % MPB, bc = e / MPB;
    const bool ok = bc < BC && mm < nm;
    pre[j] = spec[ok ? int64_t(bc) * M + mbase + mm : 0];
  }
}

template <int MPB>
__device__ __forceinline__ void put(float2* dst, const float2 (&pre)[PRE], const float2* __restrict__ spec, int BC,
                                    int64_t M, int64_t mbase, int nm) {
#pragma unroll
  for (int j = 0; j < PRE; ++j) {
    const int e = threadIdx.x + 256 * j;
    const int mm = e % MPB, bc = e / MPB;
    if (bc < BC && mm < nm) dst[sidx<MPB>(bc, mm)] = pre[j];
  }
  for (int e = threadIdx.x + 256 * PRE; e < BC * MPB; e += 256) {
    const int mm = e % MPB, bc = e / MPB;
    if (mm < nm) dst[sidx<MPB>(bc, mm)] = spec[int64_t(bc) * M + mbase + mm];
  }
}

template <int MPB>
__device__ __forceinline__ void unstage(float2* __restrict__ spec, const float2* src, int BC, int64_t M,
                                        int64_t mbase, int nm) {
  for (int e = threadIdx.x; e < BC * MPB; e += 256) {
    const int mm = e % MPB, bc = e / MPB;
    if (mm < nm) spec[int64_t(bc) * M + mbase + mm] = src[sidx<MPB>(bc, mm)];
  }
}

// Workgroups are dispatched round-robin over the 8 XCDs, each with its own
// L2.  Give each XCD a contiguous run of mode blocks, so that neighbouring
// blocks -- which read the two halves of the same 128-byte lines of the
// spectra -- share an L2 and each line is fetched from HBM once.
__device__ __forceinline__ int64_t first_block() {
  const int64_t grid = gridDim.x, bid = blockIdx.x;
  const int64_t per = grid / 8;
  if (bid >= per * 8) return bid;
  return (bid % 8) * per + bid / 8;
}

// The contiguous run of mode blocks [*k0, *k1) of this workgroup.
__device__ __forceinline__ void span(int64_t nblk, int64_t* k0, int64_t* k1) {
  *k0 = nblk * blockIdx.x / gridDim.x;
  *k1 = nblk * (blockIdx.x + 1) / gridDim.x;
}

// Loads rows i0 .. i0 + R - 1 of the (ci x co) matrix at `base` into v;
// rows or columns outside the matrix (and inactive groups) read its first
// element and are never used.
template <int OPL, int R>
__device__ __forceinline__ void load_rows(float2 (&v)[R][OPL], const float2* __restrict__ base, int i0, int ci,
                                          int co, int lr, int lpr, bool active) {
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int s = 0; s < OPL; ++s) {
      const int i = i0 + r, o = lr + lpr * s;
      const bool ok = active && i < ci && o < co;
      v[r][s] = base[ok ? int64_t(i) * co + o : 0];
    }
}

// Sum of v over each aligned group of LPR lanes (a power of two <= 64),
// with DPP steps: pairs and quads (quad_perm), 8 and 16 lanes (row half
// mirror, row mirror), then 32 and 64 lanes by broadcasting the last lane of
// a row into the next row(s).  The full sum is valid in the group's last
// lane (lanes >= 16 of a 32-lane group, >= 48 of a 64-lane group; every lane
// for groups up to 16).
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROWS, 0xf, false));
}
template <int LPR>
__device__ __forceinline__ float group_sum(float v) {
  if (LPR > 1) v += dpp<0xB1, 0xf>(v);   // quad_perm [1, 0, 3, 2]
  if (LPR > 2) v += dpp<0x4E, 0xf>(v);   // quad_perm [2, 3, 0, 1]
  if (LPR > 4) v += dpp<0x141, 0xf>(v);  // row_half_mirror
  if (LPR > 8) v += dpp<0x140, 0xf>(v);  // row_mirror
  if (LPR > 16) v += dpp<0x142, 0xa>(v); // row_bcast:15 into rows 1 and 3
  if (LPR > 32) v += dpp<0x143, 0xc>(v); // row_bcast:31 into rows 2 and 3
  return v;
}

__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
  return make_float2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
// conj(a) * b
__device__ __forceinline__ float2 cjmul(float2 a, float2 b) {
  return make_float2(a.x * b.x + a.y * b.y, a.x * b.y - a.y * b.x);
}

// mix and mix_h: one mode block per workgroup (the grid covers every
// block), in the XCD-aware order above.
template <int LPR, int OPL>
__global__ void __launch_bounds__(256)
mix_kernel(const float2* __restrict__ x, const float2* __restrict__ w, float2* __restrict__ y, MixArgs a) {
  constexpr int R = Rows<OPL>::value;
  constexpr int MPB = 256 / LPR;
  extern __shared__ float2 sm[];
  float2* sx = sm;                                // B * ci rows
  float2* sy = sm + a.B * a.ci * (MPB + 1);       // B * co rows
  const int lr = threadIdx.x % LPR, mm = threadIdx.x / LPR;
  for (int64_t k = first_block(); k < a.nblk; k += gridDim.x) {
    const int64_t lm0 = k * MPB;  // local mode index in [0, count)
    const int nm = static_cast<int>(min(int64_t(MPB), a.count - lm0));
    const int64_t mbase = a.m0 + lm0;
    const bool active = mm < nm;
    const float2* wm = w + (lm0 + (active ? mm : 0)) * int64_t(a.ci) * a.co;
    float2 wv[R][OPL];
    load_rows<OPL, R>(wv, wm, 0, a.ci, a.co, lr, LPR, active);
    stage<MPB>(sx, x, a.B * a.ci, a.M, mbase, nm);
    __syncthreads();
    for (int i0 = 0; i0 < a.ci; i0 += R) {
      if (i0 > 0) load_rows<OPL, R>(wv, wm, i0, a.ci, a.co, lr, LPR, active);
      for (int b0 = 0; b0 < a.B; b0 += BCH) {
        float2 acc[BCH][OPL];
#pragma unroll
        for (int q = 0; q < BCH; ++q)
#pragma unroll
          for (int s = 0; s < OPL; ++s) acc[q][s] = make_float2(0.f, 0.f);
#pragma unroll
        for (int r = 0; r < R; ++r) {
          if (i0 + r >= a.ci) continue;
#pragma unroll
          for (int q = 0; q < BCH; ++q) {
            if (b0 + q >= a.B) continue;
            const float2 xv = sx[sidx<MPB>((b0 + q) * a.ci + i0 + r, mm)];
#pragma unroll
            for (int s = 0; s < OPL; ++s) {
              const float2 p = cmul(xv, wv[r][s]);
              acc[q][s].x += p.x;
              acc[q][s].y += p.y;
            }
          }
        }
        if (active) {
#pragma unroll
          for (int q = 0; q < BCH; ++q) {
            if (b0 + q >= a.B) continue;
#pragma unroll
            for (int s = 0; s < OPL; ++s) {
              const int o = lr + LPR * s;
              if (o >= a.co) continue;
              float2* d = sy + sidx<MPB>((b0 + q) * a.co + o, mm);
              if (i0 > 0) {
                acc[q][s].x += d->x;
                acc[q][s].y += d->y;
              }
              *d = acc[q][s];
            }
          }
        }
      }
    }
    __syncthreads();
    unstage<MPB>(y, sy, a.B * a.co, a.M, mbase, nm);
    __syncthreads();
  }
}

// Data gradient: each row (m, i) of w gives g_x[b, i, m] for every b as a
// sum over the row's C_out columns, reduced across the row group's lanes.
template <int LPR, int OPL>
__global__ void __launch_bounds__(256)
mix_h_kernel(const float2* __restrict__ gy, const float2* __restrict__ w, float2* __restrict__ gx, MixArgs a) {
  constexpr int R = Rows<OPL>::value;
  constexpr int MPB = 256 / LPR;
  extern __shared__ float2 sm[];
  float2* sg = sm;                                // B * co rows
  float2* sx = sm + a.B * a.co * (MPB + 1);       // B * ci rows
  const int lr = threadIdx.x % LPR, mm = threadIdx.x / LPR;
  for (int64_t k = first_block(); k < a.nblk; k += gridDim.x) {
    const int64_t lm0 = k * MPB;
    const int nm = static_cast<int>(min(int64_t(MPB), a.count - lm0));
    const int64_t mbase = a.m0 + lm0;
    const bool active = mm < nm;
    const float2* wm = w + (lm0 + (active ? mm : 0)) * int64_t(a.ci) * a.co;
    float2 wv[R][OPL];
    load_rows<OPL, R>(wv, wm, 0, a.ci, a.co, lr, LPR, active);
    stage<MPB>(sg, gy, a.B * a.co, a.M, mbase, nm);
    __syncthreads();
    for (int i0 = 0; i0 < a.ci; i0 += R) {
      if (i0 > 0) load_rows<OPL, R>(wv, wm, i0, a.ci, a.co, lr, LPR, active);
      for (int b0 = 0; b0 < a.B; b0 += BCH) {
        // this lane's columns of g_y for the batch chunk
        float2 gv[BCH][OPL];
#pragma unroll
        for (int q = 0; q < BCH; ++q)
#pragma unroll
          for (int s = 0; s < OPL; ++s) {
            const int o = lr + LPR * s;
            gv[q][s] = (b0 + q < a.B && o < a.co && active) ? sg[sidx<MPB>((b0 + q) * a.co + o, mm)]
                                                             : make_float2(0.f, 0.f);
          }
#pragma unroll
        for (int r = 0; r < R; ++r) {
          if (i0 + r >= a.ci) continue;
#pragma unroll
          for (int q = 0; q < BCH; ++q) {
            if (b0 + q >= a.B) continue;
            float2 t = make_float2(0.f, 0.f);
#pragma unroll
            for (int s = 0; s < OPL; ++s) {
              const float2 p = cjmul(wv[r][s], gv[q][s]);
              t.x += p.x;
              t.y += p.y;
            }
            t.x = group_sum<LPR>(t.x);
            t.y = group_sum<LPR>(t.y);
            if (lr == LPR - 1 && active) sx[sidx<MPB>((b0 + q) * a.ci + i0 + r, mm)] = t;
          }
        }
      }
    }
    __syncthreads();
    unstage<MPB>(gx, sx, a.B * a.ci, a.M, mbase, nm);
    __syncthreads();
  }
}

// Weight gradient: a grid of resident workgroups, each walking its run of
// mode blocks.  Per block its spectra go from registers to one half of a
// double-buffered LDS area, the next block's are fetched, one barrier; then
// each lane forms its columns of a chunk of rows (m, i) in registers -- its
// g_y values of the batch chunk held in registers, x broadcast from LDS --
// and streams the rows out with non-temporal stores (g_w is written once and
// not read back here, except for the accumulate read-modify-write).  With
// almost no reads to overlap, this keeps the stores flowing while the next
// block's spectra arrive.  W = 2: every lane holds the column pairs
// o = 2 (lr + LPR s) + {0, 1} and writes them with one 16-byte store (half
// the store instructions of W = 1 for the same bytes; needs an even C_out
// and a 16-byte aligned g_w).
template <int LPR, int OPL, int W, int ACC>
__global__ void __launch_bounds__(256)
wgrad_kernel(const float2* __restrict__ x, const float2* __restrict__ gy, float2* __restrict__ gw, MixArgs a) {
  constexpr int R = Rows<OPL>::value;
  constexpr int MPB = 256 / LPR;
  extern __shared__ float2 sm[];
  const int nx = a.B * a.ci * (MPB + 1), ng = a.B * a.co * (MPB + 1);
  const int lr = threadIdx.x % LPR, mm = threadIdx.x / LPR;
  auto col = [&](int s, int w) { return W * (lr + LPR * s) + w; };
  int64_t k0, k1;
  span(a.nblk, &k0, &k1);
  float2 prex[PRE], preg[PRE];
  if (k0 < k1) {
    const int nm0 = int(min(int64_t(MPB), a.count - k0 * MPB));
    fetch<MPB>(prex, x, a.B * a.ci, a.M, a.m0 + k0 * MPB, nm0);
    fetch<MPB>(preg, gy, a.B * a.co, a.M, a.m0 + k0 * MPB, nm0);
  }
  for (int64_t k = k0; k < k1; ++k) {
    float2* sx = sm + ((k - k0) & 1) * (nx + ng);  // B * ci rows
    float2* sg = sx + nx;                          // B * co rows
    const int64_t lm0 = k * MPB;
    const int nm = static_cast<int>(min(int64_t(MPB), a.count - lm0));
    const int64_t mbase = a.m0 + lm0;
    const bool active = mm < nm;
    float2* gm = gw + (lm0 + (active ? mm : 0)) * int64_t(a.ci) * a.co;
    // rows i0 .. i0 + R - 1 of this mode's (ci x co) block of g_w (the
    // accumulate read; rows or columns outside read its first element and
    // are never used)
    auto load_acc = [&](float2 (&v)[R][OPL][W], int i0) {
#pragma unroll
      for (int r = 0; r < R; ++r)
#pragma unroll
        for (int s = 0; s < OPL; ++s) {
          const int i = i0 + r, o = col(s, 0);
          const bool ok = active && i < a.ci && o < a.co;
          const float2* src = gm + (ok ? int64_t(i) * a.co + o : 0);
          if (W == 2) {
            const float4 t = *reinterpret_cast<const float4*>(src);
            v[r][s][0] = make_float2(t.x, t.y);
            v[r][s][W - 1] = make_float2(t.z, t.w);
          } else {
            v[r][s][0] = *src;
          }
        }
    };
    float2 acc[R][OPL][W];
    if constexpr (ACC) load_acc(acc, 0);
    put<MPB>(sx, prex, x, a.B * a.ci, a.M, mbase, nm);
    put<MPB>(sg, preg, gy, a.B * a.co, a.M, mbase, nm);
    if (k + 1 < k1) {
      const int nm1 = int(min(int64_t(MPB), a.count - lm0 - MPB));
      fetch<MPB>(prex, x, a.B * a.ci, a.M, mbase + MPB, nm1);
      fetch<MPB>(preg, gy, a.B * a.co, a.M, mbase + MPB, nm1);
    }
    __syncthreads();
    if (!active) continue;
    for (int i0 = 0; i0 < a.ci; i0 += R) {
      if constexpr (ACC) {
        if (i0 > 0) load_acc(acc, i0);
      } else {
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
          for (int s = 0; s < OPL; ++s)
#pragma unroll
            for (int w = 0; w < W; ++w) acc[r][s][w] = make_float2(0.f, 0.f);
      }
      for (int b0 = 0; b0 < a.B; b0 += BCH) {
        float2 gv[BCH][OPL][W];
#pragma unroll
        for (int q = 0; q < BCH; ++q)
#pragma unroll
          for (int s = 0; s < OPL; ++s)
#pragma unroll
            for (int w = 0; w < W; ++w) {
              const int o = col(s, w);
              gv[q][s][w] =
                  (b0 + q < a.B && o < a.co) ? sg[sidx<MPB>((b0 + q) * a.co + o, mm)] : make_float2(0.f, 0.f);
            }
#pragma unroll
        for (int r = 0; r < R; ++r) {
          if (i0 + r >= a.ci) continue;
#pragma unroll
          for (int q = 0; q < BCH; ++q) {
            if (b0 + q >= a.B) continue;
            const float2 xv = sx[sidx<MPB>((b0 + q) * a.ci + i0 + r, mm)];
#pragma unroll
            for (int s = 0; s < OPL; ++s)
#pragma unroll
              for (int w = 0; w < W; ++w) {
                const float2 p = cjmul(xv, gv[q][s][w]);
                acc[r][s][w].x += p.x;
                acc[r][s][w].y += p.y;
              }
          }
        }
      }
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int i = i0 + r;
        if (i >= a.ci) continue;
#pragma unroll
        for (int s = 0; s < OPL; ++s) {
          const int o = col(s, 0);
          if (o >= a.co) continue;
          if (W == 2)
            __builtin_nontemporal_store(v4f{acc[r][s][0].x, acc[r][s][0].y, acc[r][s][W - 1].x, acc[r][s][W - 1].y},
                                        reinterpret_cast<v4f*>(gm + int64_t(i) * a.co + o));
          else
            __builtin_nontemporal_store(v2f{acc[r][s][0].x, acc[r][s][0].y},
                                        reinterpret_cast<v2f*>(gm + int64_t(i) * a.co + o));
        }
      }
    }
  }
}

int lanes_per_row(int64_t co) {
  int l = 1;
  while (l < co && l < 64) l <<= 1;
  return l;
}

int opl_of(int64_t co) {
  const int64_t o = (co + 63) / 64;
  return o <= 1 ? 1 : (o <= 2 ? 2 : (o <= 4 ? 4 : 8));
}

// cols: the columns one lane group spans per row slot (C_out, or C_out / 2
// for wgrad's column pairs).
MixArgs make_args(int64_t B, int64_t ci, int64_t co, int64_t M, int64_t m0, int64_t m1, int acc,
                  int64_t cols = 0) {
  MixArgs a;
  a.M = M;
  a.m0 = m0;
  a.count = m1 - m0;
  a.B = static_cast<int>(B);
  a.ci = static_cast<int>(ci);
  a.co = static_cast<int>(co);
  a.lpr = lanes_per_row(cols > 0 ? cols : co);
  a.mpb = 256 / a.lpr;
  a.acc = acc;
  a.nblk = (a.count + a.mpb - 1) / a.mpb;
  return a;
}

typedef void (*mix_fn)(const float2*, const float2*, float2*, MixArgs);

// Workgroups of kernel f with `lds` bytes of LDS the current device holds at
// once (cached per kernel, LDS size and device).
int64_t resident_workgroups(mix_fn f, size_t lds) {
  struct Entry {
    mix_fn f;
    size_t lds;
    int dev;
    int64_t n;
  };
  static std::mutex mu;
  static std::vector<Entry> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  {
    std::lock_guard<std::mutex> lock(mu);
    for (const Entry& e : cache)
      if (e.f == f && e.lds == lds && e.dev == dev) return e.n;
  }
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, f, 256, lds) != hipSuccess) return 0;
  const int64_t n = int64_t(cus) * (per_cu > 0 ? per_cu : 1);
  std::lock_guard<std::mutex> lock(mu);
  cache.push_back(Entry{f, lds, dev, n});
  return n;
}

// LDS of one mode block's spectra (mode blocks of 256 / lanes_per_row(cols)
// modes; cols = C_out unless given).
size_t block_lds(int64_t B, int64_t ci, int64_t co, int64_t cols = 0) {
  const size_t mpb = size_t(256 / lanes_per_row(cols > 0 ? cols : co));
  return sizeof(float2) * size_t(B) * size_t(ci + co) * (mpb + 1);
}

// persistent: a grid of resident workgroups walking runs of blocks (wgrad);
// else one workgroup per block (capped at 2^22, the kernels loop beyond).
int launch(mix_fn f, size_t lds, bool persistent, const float2* p0, const float2* p1, float2* p2, const MixArgs& a,
           void* stream) {
  if (lds > 65536) {
    const hipError_t e =
        hipFuncSetAttribute(reinterpret_cast<const void*>(f), hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
    if (e != hipSuccess) return e;
  }
  int64_t cap = int64_t(1) << 22;
  if (persistent) {
    cap = resident_workgroups(f, lds);
    if (cap <= 0) return hipErrorInvalidConfiguration;
  }
  const int64_t blocks = a.nblk < cap ? a.nblk : cap;
  hipLaunchKernelGGL(f, dim3(static_cast<unsigned>(blocks)), dim3(256), lds, static_cast<hipStream_t>(stream), p0,
                     p1, p2, a);
  return hipGetLastError();
}

}  // namespace

// LDS a mix workgroup needs: wgrad's double-buffered spectra of one mode
// block (mix and mix_h use half of it; wgrad's column-pair form, taken only
// where it fits, twice as many modes).
size_t mix_lds_bytes(int64_t B, int64_t ci, int64_t co) { return 2 * block_lds(B, ci, co); }

namespace {

// Kernel instance for C_out: LPR lanes per row and OPL columns per lane.
template <template <int, int> class K>
mix_fn pick(int64_t co) {
  switch (lanes_per_row(co)) {
    case 1: return K<1, 1>::fn;
    case 2: return K<2, 1>::fn;
    case 4: return K<4, 1>::fn;
    case 8: return K<8, 1>::fn;
    case 16: return K<16, 1>::fn;
    case 32: return K<32, 1>::fn;
    default: break;
  }
  const int opl = opl_of(co);
  return opl == 1 ? K<64, 1>::fn : opl == 2 ? K<64, 2>::fn : opl == 4 ? K<64, 4>::fn : K<64, 8>::fn;
}
template <int L, int O>
struct MixK {
  static constexpr mix_fn fn = mix_kernel<L, O>;
};
template <int L, int O>
struct MixHK {
  static constexpr mix_fn fn = mix_h_kernel<L, O>;
};
// (accumulating and overwriting instances apart: the accumulate read and its
// conditions are not compiled into the overwriting kernel)
template <int L, int O>
struct WgradK {
  static constexpr mix_fn fn = wgrad_kernel<L, O, 1, 0>;
};
template <int L, int O>
struct WgradK2 {
  static constexpr mix_fn fn = wgrad_kernel<L, O, 2, 0>;
};
template <int L, int O>
struct WgradKA {
  static constexpr mix_fn fn = wgrad_kernel<L, O, 1, 1>;
};
template <int L, int O>
struct WgradK2A {
  static constexpr mix_fn fn = wgrad_kernel<L, O, 2, 1>;
};

}  // namespace

int launch_mix(const void* xhat, const void* w, void* yhat, int64_t B, int64_t ci, int64_t co, int64_t M,
               int64_t m0, int64_t m1, void* stream) {
  if (B <= 0 || m1 <= m0) return hipSuccess;
  const MixArgs a = make_args(B, ci, co, M, m0, m1, 0);
  return launch(pick<MixK>(co), block_lds(B, ci, co), false, static_cast<const float2*>(xhat),
                static_cast<const float2*>(w), static_cast<float2*>(yhat), a, stream);
}

int launch_mix_h(const void* gy, const void* w, void* gx, int64_t B, int64_t ci, int64_t co, int64_t M,
                 int64_t m0, int64_t m1, void* stream) {
  if (B <= 0 || m1 <= m0) return hipSuccess;
  const MixArgs a = make_args(B, ci, co, M, m0, m1, 0);
  return launch(pick<MixHK>(co), block_lds(B, ci, co), false, static_cast<const float2*>(gy),
                static_cast<const float2*>(w), static_cast<float2*>(gx), a, stream);
}

int launch_wgrad(const void* xhat, const void* gy, void* gw, int64_t B, int64_t ci, int64_t co, int64_t M,
                 int64_t m0, int64_t m1, int accumulate, void* stream) {
  if (B <= 0 || m1 <= m0) return hipSuccess;
  // column pairs (16-byte stores) for an even C_out of at least 4 when g_w
  // is 16-byte aligned and the doubled mode block still fits the LDS
  const size_t lds2 = 2 * block_lds(B, ci, co, co / 2);
  if (co % 2 == 0 && co >= 4 && (reinterpret_cast<uintptr_t>(gw) & 15) == 0 && lds2 <= 160 * 1024) {
    const MixArgs a = make_args(B, ci, co, M, m0, m1, accumulate ? 1 : 0, co / 2);
    return launch(accumulate ? pick<WgradK2A>(co / 2) : pick<WgradK2>(co / 2), lds2, true,
                  static_cast<const float2*>(xhat),
                  static_cast<const float2*>(gy), static_cast<float2*>(gw), a, stream);
  }
  const MixArgs a = make_args(B, ci, co, M, m0, m1, accumulate ? 1 : 0);
  return launch(accumulate ? pick<WgradKA>(co) : pick<WgradK>(co), mix_lds_bytes(B, ci, co), true,
                static_cast<const float2*>(xhat),
                static_cast<const float2*>(gy), static_cast<float2*>(gw), a, stream);
}

}  // namespace dtst
