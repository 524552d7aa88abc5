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

#include <type_traits>

#include "dtst_internal.h"

namespace dtst {
namespace {

#include "stream_ops.h"


// ---------------------------------------------------------------------------
// Forward: x (rows x N_z x N_t) fp32 -> out (rows x K_z x K_t) complex.
//
// A row is taken in z tiles (16 z per class).  load_tile fetches one tile,
// tz_tile contracts its t then z into the row's accumulators, and tz_finish
// turns the accumulators of a finished row into complex coefficients.
// MODE 0: scalar loads (N_t % 4 != 0); 1: 16-byte loads with masks;
// 2: 16-byte loads of complete tiles, no masks.  Loads are unconditional
// (out-of-range lanes read the row start) and masked when the values are
// used, so nothing between the loads and the MFMAs forces an early wait.
// ---------------------------------------------------------------------------
template <int TH, int NCLS, int MODE>
__device__ __forceinline__ void load_tile(const float* __restrict__ x, const StreamArgs& a, int m, int g, int64_t r,
                                          int zt, float (&dst)[NCLS][TH][4], bool (&ok)[NCLS][TH * 4]) {
  const float* xr = x + r * (int64_t(a.nz) * a.nt);
  const int zl = zt * 16 + m;
  const bool zok = zl < a.zh;
#pragma unroll
  for (int hf = 0; hf < NCLS; ++hf) {
    const int64_t zoff = int64_t(zl + hf * a.zh) * a.nt;
#pragma unroll
    for (int h = 0; h < TH; ++h) {
      if (MODE == 2) {
        const float4 v = *reinterpret_cast<const float4*>(xr + zoff + 16 * h + 4 * g);
        dst[hf][h][0] = v.x; dst[hf][h][1] = v.y; dst[hf][h][2] = v.z; dst[hf][h][3] = v.w;
        ok[hf][4 * h] = true;
      } else if (MODE == 1) {
        const int t0 = 16 * h + 4 * g;
        const bool v_ok = zok && t0 < a.nt;
        const float4 v = *reinterpret_cast<const float4*>(xr + (v_ok ? zoff + t0 : 0));
        dst[hf][h][0] = v.x; dst[hf][h][1] = v.y; dst[hf][h][2] = v.z; dst[hf][h][3] = v.w;
        ok[hf][4 * h] = v_ok;
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int t = 16 * h + 4 * g + j;
          const bool v_ok = zok && t < a.nt;
          dst[hf][h][j] = xr[v_ok ? zoff + t : 0];
          ok[hf][4 * h + j] = v_ok;
        }
      }
    }
  }
}

// Contracts t of the tile held in xv (z = 16zt + m and the partner z of
// every other class) into V, then folds the classes.  With TF the lane's
// t and t + N_t/2 (groups h and h + TH/2) are combined first; only the
// first 4 TH / 2 steps of bt are used then.
template <int CT, int TH, int NCLS, int MODE, int TF = 0>
__device__ __forceinline__ void t_part(const float (&xv)[NCLS][TH][4], const bool (&ok)[NCLS][TH * 4],
                                       const float (&bt)[TH * 4][CT], v4f (&V)[NCLS][CT]) {
#pragma unroll
  for (int hf = 0; hf < NCLS; ++hf)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) V[hf][ct] = v4f{0.f, 0.f, 0.f, 0.f};
  if constexpr (TF) {
    static_assert(CT == 2 && TH % 2 == 0 && MODE != 0, "t folding needs two k_t tiles and whole 16-byte t groups");
#pragma unroll
    for (int h = 0; h < TH / 2; ++h)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int hf = 0; hf < NCLS; ++hf) {
          const float lo = (MODE == 2 || ok[hf][4 * h]) ? xv[hf][h][j] : 0.f;
          const float hi = (MODE == 2 || ok[hf][4 * (h + TH / 2)]) ? xv[hf][h + TH / 2][j] : 0.f;
          V[hf][0] = mfma(lo + hi, bt[h * 4 + j][0], V[hf][0]);
          V[hf][1] = mfma(lo - hi, bt[h * 4 + j][1], V[hf][1]);
        }
    fold_classes<NCLS, CT, TF>(V);
    return;
  }
#pragma unroll
  for (int h = 0; h < TH; ++h)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int hf = 0; hf < NCLS; ++hf) {
        const float xa = (MODE == 2 || ok[hf][MODE == 1 ? 4 * h : 4 * h + j]) ? xv[hf][h][j] : 0.f;
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) V[hf][ct] = mfma(xa, bt[h * 4 + j][ct], V[hf][ct]);
      }
  fold_classes<NCLS, CT>(V);
}

// Contracts z of the t-contracted tile V (z tile zt) into P; P is cleared
// first when zt == 0.  Accumulator register i of V is the B operand of the
// step whose K index is z = 16zt + 4g + i.
//
// t-folded (TF) tiles take the complex product in three real products
// instead of four: with B = Br + i Bi and V = Vr + i Vi,
//   k1 = Br (Vr + Vi),   k2 = (Bi - Br) Vr,   k3 = (Br + Bi) Vi,
//   Re BV = k1 - k3,     Im BV = k1 + k2,
// the three basis factors read from the image (blocks mr, mr + MT/2 and
// mr + MT of a class and z tile), accumulated in P[.][mr][0] (k1),
// P[.][mr][1] (k2) and P[.][mr + MT/2][0] (k3).  The B operands are
// rearranged first so that lanes m < 8 carry the even k_t = 2m and lanes
// m >= 8 the odd k_t = 2(m - 8) + 1 (Re and Im then share a lane and the
// finish needs no exchange).
template <int CT, int MT, int NCLS, int TF = 0>
__device__ __forceinline__ void z_part(const v4f (&V)[NCLS][CT], const float4* lds, const StreamArgs& a, int zt,
                                       int lane, v4f (&P)[NCLS][MT][CT]) {
  constexpr int MTS = TF ? 3 * MT / 2 : MT;  // image blocks per (class, z tile)
  float4 A[NCLS][MT];
#pragma unroll
  for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) A[cl][mt] = lds[((cl * a.zt + zt) * MTS + mt) * 64 + lane];
  if (zt == 0) {
#pragma unroll
    for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) P[cl][mt][ct] = v4f{0.f, 0.f, 0.f, 0.f};
  }
  if constexpr (TF) {
    static_assert(CT == 2 && MT % 2 == 0, "t-folded tiles: two k_t tiles, Re and Im row tiles");
    // image blocks per (class, z tile): Br, Bi - Br and Br + Bi row tiles
    constexpr int MTI = 3 * MT / 2;
    float4 Bs[NCLS][MT / 2];
#pragma unroll
    for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
      for (int mr = 0; mr < MT / 2; ++mr) Bs[cl][mr] = lds[((cl * a.zt + zt) * MTI + MT + mr) * 64 + lane];
    v4f G1[NCLS], G2[NCLS], G3[NCLS];
#pragma unroll
    for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        // tile 0: Re (m < 8) / Im (m >= 8) of even k_t; tile 1: the same of odd k_t
        const float t0 = V[cl][0][i], t1 = V[cl][1][i];
        // Im V of this lane's k_t: lanes m < 8 take lane m + 8 of tile 0
        // (DPP banks 0, 1), lanes m >= 8 keep tile 1; Re V: lanes m >= 8 take
        // lane m - 8 of tile 1 (banks 2, 3), lanes m < 8 keep tile 0
        const float vi = ror8_into<0x3>(t1, t0);
        const float vr = ror8_into<0xC>(t0, t1);
        G1[cl][i] = vr + vi;
        G2[cl][i] = vr;
        G3[cl][i] = vi;
      }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
        for (int mr = 0; mr < MT / 2; ++mr) {
          // A[.][mr] = Br, A[.][mr + MT/2] = Bi - Br, Bs = Br + Bi
          P[cl][mr][0] = mfma(A[cl][mr][i], G1[cl][i], P[cl][mr][0]);
          P[cl][mr][1] = mfma(A[cl][mr + MT / 2][i], G2[cl][i], P[cl][mr][1]);
          P[cl][mr + MT / 2][0] = mfma(Bs[cl][mr][i], G3[cl][i], P[cl][mr + MT / 2][0]);
        }
    return;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) P[cl][mt][ct] = mfma(A[cl][mt][i], V[cl][ct][i], P[cl][mt][ct]);
}

// Combines the real-stacked products of a finished row into complex
// coefficients and hands each one to st(index p * K_t + k_t, re, im):
// (Re B) V and (Im B) V sit in row tiles mt and mt + MT/2 of the same lane;
// the Re / Im columns of k_t sit 8 lanes apart (CT = 1, and CT = 2 with TF)
// or in the two column tiles (CT = 2).
template <int CT, int MT, int NCLS, int TF = 0, class Store>
__device__ __forceinline__ void tz_finish(const v4f (&P)[NCLS][MT][CT], const StreamArgs& a, int m, int g,
                                          Store&& st) {
  constexpr int KTP = 8 * CT;
  if constexpr (TF) {
    // Lanes m < 8 hold the even k_t = 2m, lanes m >= 8 the odd
    // k_t = 2(m - 8) + 1 (three-product form of z_part):
    // Re = k1 - k3, Im = k1 + k2.
    const bool hi = m >= 8;
    const int kc = 2 * (m & 7) + (hi ? 1 : 0);
#pragma unroll
    for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
      for (int mr = 0; mr < MT / 2; ++mr)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float k1 = P[cl][mr][0][i], k2 = P[cl][mr][1][i], k3 = P[cl][mr + MT / 2][0][i];
          const int p = (16 * mr + 4 * g + i) * NCLS + cl;
          if (kc < a.kt && p < a.kz) st(p * a.kt + kc, k1 - k3, k1 + k2);
        }
  } else if constexpr (CT == 1 && MT == 1) {
    static_assert(NCLS == 4, "one row tile per class is used by the four-class z fold only");
    // Register 2j holds (Re B) V and register 2j + 1 (Im B) V of slot
    // s = 2g + j.  Lanes m < 8 finish class 2cp (k_t = m), lanes m >= 8
    // class 2cp + 1 (k_t = m - 8) of the same slot, trading values as below;
    // the two modes 4s + 2cp and 4s + 2cp + 1 are adjacent.
    const bool hi = m >= KTP;
    const int kc = hi ? m - KTP : m;
#pragma unroll
    for (int cp = 0; cp < NCLS / 2; ++cp)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const float q0 = P[2 * cp][0][0][2 * j], u0 = P[2 * cp][0][0][2 * j + 1];
        const float q1 = P[2 * cp + 1][0][0][2 * j], u1 = P[2 * cp + 1][0][0][2 * j + 1];
        const float rq = ror8(hi ? q0 : q1);
        const float ru = ror8(hi ? u0 : u1);
        const float re = hi ? rq - u1 : q0 - ru;
        const float im = hi ? q1 + ru : rq + u0;
        const int p = (2 * g + j) * NCLS + 2 * cp + (hi ? 1 : 0);
        if (kc < a.kt && p < a.kz) st(p * a.kt + kc, re, im);
      }
  } else if constexpr (CT == 1) {
    static_assert(NCLS <= 2, "the four-class z fold of one column tile uses one row tile per class");
    // Lanes m < 8 finish mode p0 (k_t = m), lanes m >= 8 the next mode
    // p0 + 1 (k_t = m - 8): z class 1 of the same slot when folded, else
    // the next accumulator register.  Each lane pair trades the values the
    // other half needs, so every store instruction covers whole 128-byte
    // rows of two adjacent modes.
    const bool hi = m >= KTP;
    const int kc = hi ? m - KTP : m;
#pragma unroll
    for (int mr = 0; mr < MT / 2; ++mr)
#pragma unroll
      for (int j = 0; j < (NCLS == 2 ? 4 : 2); ++j) {
        const int i0 = NCLS == 2 ? j : 2 * j, i1 = NCLS == 2 ? j : 2 * j + 1;
        const int c1 = NCLS - 1;
        const float q0 = P[0][mr][0][i0], u0 = P[0][mr + MT / 2][0][i0];
        const float q1 = P[c1][mr][0][i1], u1 = P[c1][mr + MT / 2][0][i1];
        const float rq = ror8(hi ? q0 : q1);
        const float ru = ror8(hi ? u0 : u1);
        const float re = hi ? rq - u1 : q0 - ru;
        const float im = hi ? q1 + ru : rq + u0;
        const int p = (NCLS == 2 ? 2 * (16 * mr + 4 * g + i0) : 16 * mr + 4 * g + i0) + (hi ? 1 : 0);
        if (kc < a.kt && p < a.kz) st(p * a.kt + kc, re, im);
      }
  } else {
#pragma unroll
    for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
      for (int mr = 0; mr < MT / 2; ++mr)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int p = (16 * mr + 4 * g + i) * NCLS + cl;
          const float rr = P[cl][mr][0][i], ri = P[cl][mr][CT - 1][i];
          const float ir = P[cl][mr + MT / 2][0][i], ii = P[cl][mr + MT / 2][CT - 1][i];
          if (m < a.kt && p < a.kz) st(p * a.kt + m, rr - ii, ri + ir);
        }
  }
}

// Every wave walks its (row, z-tile) pairs in order and keeps the next PD
// pairs' loads in flight while it computes the current one (PD = 2 for the
// t-folded instances, whose tiles take the fewest products per byte, else
// 1).  Buffer k holds the tiles k, k + PD, k + 2 PD, ... and is refilled as
// soon as its tile is contracted; the loop runs whole passes over the PD
// buffers so that every buffer index is a compile-time constant (no
// register copies, which would wait for loads still in flight).  Every load
// is unconditional -- positions past the wave's last tile re-read its last
// row and are never contracted -- so that the wait for a tile covers that
// tile's loads only, not the ones issued after it.
template <int CT, int TH, int MT, int NCLS, int MODE, int TF>
__device__ __forceinline__ void fwd_tz_body(const float* __restrict__ x, float2* __restrict__ out,
                                            const float (&bt)[TH * 4][CT], const float4* lds,
                                            const StreamArgs& a, int64_t wave, int64_t wstride) {
  constexpr int PD = TF ? 2 : 1;
  const int lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int64_t n_rows = (a.rows - 1 - wave) / wstride + 1;
  const int64_t n_iter = n_rows * a.zt;
  const int64_t last_row = wave + (n_rows - 1) * wstride;

  float xb[PD][NCLS][TH][4];
  bool okb[PD][NCLS][TH * 4];
  int64_t rp[PD], itp[PD];
  int ztp[PD];
  int64_t rn = wave, itn = 0;
  int ztn = 0;
  auto fetch = [&](int k) __attribute__((always_inline)) {
    rp[k] = rn;
    ztp[k] = ztn;
    itp[k] = itn++;
    load_tile<TH, NCLS, MODE>(x, a, m, g, rn < last_row ? rn : last_row, ztn, xb[k], okb[k]);
    if (++ztn == a.zt) {
      ztn = 0;
      rn += wstride;
    }
  };
#pragma unroll
  for (int k = 0; k < PD; ++k) fetch(k);
  v4f P[NCLS][MT][CT];

  auto step = [&](auto kc) __attribute__((always_inline)) {
    constexpr int k = decltype(kc)::value;
    const bool live = itp[k] < n_iter;
    const int64_t r = rp[k];
    const int zt = ztp[k];
    v4f V[NCLS][CT];
    if (live) t_part<CT, TH, NCLS, MODE, TF>(xb[k], okb[k], bt, V);
    fetch(k);
    if (!live) return;
    z_part<CT, MT, NCLS, TF>(V, lds, a, zt, lane, P);
    if (zt != a.zt - 1) return;
    float2* orow = out + r * int64_t(a.kz) * a.kt;
    tz_finish<CT, MT, NCLS, TF>(P, a, m, g, [&](int idx, float re, float im) { orow[idx] = make_float2(re, im); });
  };
  static_assert(PD == 1 || PD == 2, "one or two tiles in flight");
  do {
    step(std::integral_constant<int, 0>{});
    if constexpr (PD > 1) step(std::integral_constant<int, 1>{});
  } while (itp[0] < n_iter);
}

// ---------------------------------------------------------------------------
// Forward t + z + y in one pass (used when the y contraction fits: K_t <= 8,
// at most 16 z modes per class, K_y <= 32, K_z K_t <= 256).
//
// A workgroup of 16 waves owns one (b, c, x) plane at a time (persistent over
// planes).  The plane's y rows come in groups of 16 slots: with y folded (the
// shard holds the whole even N_y) a slot is the row pair (y, y + N_y/2),
// otherwise a single row.  Wave w contracts t and z of the row(s) of slot w
// exactly as fwd_tz_body does and leaves the (K_z x K_t) results in LDS.
// After a barrier, wave w < ceil(K_z K_t / 16) contracts y for the columns
// 16w..16w+15 of every slot of the group (the slots are the MFMA K index, the
// y basis image of the separate y contraction supplies the A operand; folded,
// even modes take the pair's sum and odd modes its difference), accumulating
// over the plane's groups in registers; a second barrier frees the LDS rows.
// The (K_y x K_z K_t) result of the plane is written once.  The shard is read
// once and the (N_y x K_z K_t) intermediate never reaches HBM.
// ---------------------------------------------------------------------------
// Waves per workgroup and tile buffers per wave of fwd_tzy_kernel (a tile of
// the four-class z fold is twice as large: three buffers keep two 8 KiB tiles
// in flight per wave within the registers of two waves per SIMD).
constexpr int kFusedWaves = 8;
constexpr int kFusedBufs = 4;
constexpr int kFusedBufs4 = 3;
// Staging of the fused kernels' basis images in LDS: entries [0, nimg) of
// the staged range are the z image, the next ny4 the y image, which sits
// yshift float4 further on in LDS (after the row exchange).  The copy runs in
// passes of four float4 per thread.  stage_begin copies every pass but the
// last and issues the last pass's loads; the caller then issues its own
// first loads and calls stage_end, whose LDS stores wait only for the
// staging loads (the memory counter retires loads in order), so the
// caller's loads stay in flight across the barrier that follows.  Lanes past
// the end copy the last entry again (the same value to the same address),
// so no pass has a branch.
struct StageLast {
  float4 v0, v1, v2, v3;
  int d0, d1, d2, d3;
};

__device__ __forceinline__ StageLast stage_begin(float4* lds, const float4* __restrict__ zimg,
                                                 const float4* __restrict__ yimg, int nimg, int ny4, int yshift) {
  const int tot = nimg + ny4;
  const int bd = static_cast<int>(blockDim.x), tid = static_cast<int>(threadIdx.x);
  auto src_of = [&](int i) { return i < nimg ? zimg[i] : yimg[i - nimg]; };
  auto dst_of = [&](int i) { return i < nimg ? i : i + yshift; };
  const int full = (tot - 1) / (4 * bd);
#pragma unroll 1
  for (int p = 0; p < full; ++p) {
    const int i0 = 4 * p * bd + tid;
    const float4 v0 = src_of(i0), v1 = src_of(i0 + bd), v2 = src_of(i0 + 2 * bd), v3 = src_of(i0 + 3 * bd);
    lds[dst_of(i0)] = v0;
    lds[dst_of(i0 + bd)] = v1;
    lds[dst_of(i0 + 2 * bd)] = v2;
    lds[dst_of(i0 + 3 * bd)] = v3;
  }
  const int l0 = 4 * full * bd + tid;
  const int i0 = min(l0, tot - 1), i1 = min(l0 + bd, tot - 1), i2 = min(l0 + 2 * bd, tot - 1),
            i3 = min(l0 + 3 * bd, tot - 1);
  StageLast r;
  r.v0 = src_of(i0);
  r.v1 = src_of(i1);
  r.v2 = src_of(i2);
  r.v3 = src_of(i3);
  r.d0 = dst_of(i0);
  r.d1 = dst_of(i1);
  r.d2 = dst_of(i2);
  r.d3 = dst_of(i3);
  // Keep the scheduler from moving the caller's loads above these.
  __builtin_amdgcn_sched_barrier(0);
  return r;
}

__device__ __forceinline__ void stage_end(float4* lds, const StageLast& r) {
  lds[r.d0] = r.v0;
  lds[r.d1] = r.v1;
  lds[r.d2] = r.v2;
  lds[r.d3] = r.v3;
}

struct FusedArgs {
  int64_t planes;  // B * C * N_x
  int ny;          // local N_y (rows per plane)
  int slots;       // slots per plane: N_y / 2 folded, else N_y
  int half;        // N_y / 2 folded (second row of a slot), else 0
  int jq;          // groups of 16 slots per plane
  int kth;         // k tiles per y class in the y image
  int ky;          // K_y
  int mcols;       // K_z * K_t
  int mrow;        // LDS row stride in complex values
  int nwy;         // waves running the y contraction: ceil(mcols / 16)
  int yimg_n4;     // float4 entries of the y image (staged in LDS when the kernel's YL is 1)
};

template <int TH, int NCLS, int MODE, int NCY, int KYT, int NW, int NB, int YL>
__global__ void __launch_bounds__(64 * NW)
fwd_tzy_kernel(const float* __restrict__ x, float2* __restrict__ out, const float* __restrict__ timg,
               const float4* __restrict__ zimg, const float4* __restrict__ yimg, StreamArgs a, FusedArgs f) {
  constexpr int CT = 1, MT = NCLS == 4 ? 1 : 2;
  constexpr int SPW = 16 / NW;  // slots of a group per wave
  constexpr int MTW = 16 / NW;  // 16-column tiles of the y contraction per wave
  extern __shared__ float4 lds[];
  const int nimg = NCLS * a.zt * MT * 64;
  float2* vlds = reinterpret_cast<float2*>(lds + nimg);
  const int lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int w = threadIdx.x >> 6;
  if (blockIdx.x >= f.planes) return;  // the host never launches more workgroups than planes

  // Position of a tile: (plane, slot group, slot of this wave, row of the
  // slot, z tile), z tile fastest.
  struct Cur {
    int64_t pl;
    int q, j, h, zt;
  };
  auto advance = [&](Cur c) {
    if (++c.zt == a.zt) {
      c.zt = 0;
      if (++c.h == NCY) {
        c.h = 0;
        if (++c.j == SPW) {
          c.j = 0;
          if (++c.q == f.jq) {
            c.q = 0;
            c.pl += gridDim.x;
          }
        }
      }
    }
    return c;
  };
  // Row of a tile for this wave; slots past the plane's end read its first
  // row and contribute zeros, and positions past the last plane (loaded but
  // never contracted) read the last plane.  Every load is unconditional: a
  // load behind a branch would make the compiler wait for all outstanding
  // loads (one memory counter) before each tile instead of for that tile's.
  auto row_of = [&](const Cur& c, bool* valid) {
    const int s = 16 * c.q + w + NW * c.j;
    *valid = s < f.slots;
    const int64_t pl = c.pl < f.planes ? c.pl : f.planes - 1;
    return pl * f.ny + (*valid ? s + c.h * f.half : 0);
  };

  // NB tile buffers: buffer k holds the tile at cb[k] and is refilled, once
  // contracted, with the tile NB positions further on, so NB - 1 tiles are in
  // flight while one is contracted.
  float xb[NB][NCLS][TH][4];
  bool okb[NB][NCLS][TH * 4];
  bool vb[NB];
  Cur cb[NB];
  cb[0] = Cur{static_cast<int64_t>(blockIdx.x), 0, 0, 0, 0};
#pragma unroll
  for (int k = 1; k < NB; ++k) cb[k] = advance(cb[k - 1]);
#pragma unroll
  for (int k = 0; k < NB; ++k) vb[k] = false;

  // LDS: z image, the exchanged row results, the y image (YL = 1; with
  // YL = 0 the y image is read from global memory).  The staging loads go
  // out first, then the t basis and all NB tiles; the tile loop then starts
  // with every buffer in flight, the same outstanding loads as at the end of
  // each of its passes.
  float4* ylds = reinterpret_cast<float4*>(vlds + 16 * NCY * f.mrow);
  const StageLast stl = stage_begin(lds, zimg, yimg, nimg, YL ? f.yimg_n4 : 0, 8 * NCY * f.mrow);
  // B operand of the t contraction.
  float bt[TH * 4][CT];
#pragma unroll
  for (int st = 0; st < TH * 4; ++st) bt[st][0] = timg[st * 64 + lane];
#pragma unroll
  for (int k = 0; k < NB; ++k) load_tile<TH, NCLS, MODE>(x, a, m, g, row_of(cb[k], &vb[k]), cb[k].zt, xb[k], okb[k]);
  stage_end(lds, stl);
  __syncthreads();

  v4f yr[NCY][KYT][MTW], yi[NCY][KYT][MTW];
#pragma unroll
  for (int c = 0; c < NCY; ++c)
#pragma unroll
    for (int k = 0; k < KYT; ++k)
#pragma unroll
      for (int t = 0; t < MTW; ++t) {
        yr[c][k][t] = v4f{0.f, 0.f, 0.f, 0.f};
        yi[c][k][t] = v4f{0.f, 0.f, 0.f, 0.f};
      }
  v4f P[NCLS][MT][CT];

  // Contract buffer k's tile and refill the buffer; at a row's end leave its
  // results in LDS, and after the wave's last row of a slot group run the
  // group's y contraction.
  // Tiles past the last plane (live = false, the same for the whole
  // workgroup) are loaded but not contracted.
  auto process = [&](int k) __attribute__((always_inline)) {
    const Cur c = cb[k];
    const bool valid = vb[k];
    const bool live = c.pl < f.planes;
    v4f V[NCLS][CT];
    if (live) t_part<CT, TH, NCLS, MODE>(xb[k], okb[k], bt, V);
    const Cur far = advance(cb[(k + NB - 1) % NB]);
    cb[k] = far;
    load_tile<TH, NCLS, MODE>(x, a, m, g, row_of(far, &vb[k]), far.zt, xb[k], okb[k]);
    if (!live) return;
    z_part<CT, MT, NCLS>(V, lds, a, c.zt, lane, P);
    if (c.zt != a.zt - 1) return;
    float2* vrow = vlds + (c.h * 16 + w + NW * c.j) * f.mrow;
    tz_finish<CT, MT, NCLS>(P, a, m, g, [&](int idx, float re, float im) {
      vrow[idx] = valid ? make_float2(re, im) : make_float2(0.f, 0.f);
    });
    if (c.h != NCY - 1 || c.j != SPW - 1) return;
    __syncthreads();
    float4 br[NCY][KYT], bi[NCY][KYT];
#pragma unroll
    for (int cl = 0; cl < NCY; ++cl)
#pragma unroll
      for (int kk = 0; kk < KYT; ++kk) {
        const int kt = NCY == 2 ? cl * f.kth + kk : kk;
        const int e = (kt * f.jq + c.q) * 2 * 64 + lane;
        if constexpr (YL) {
          br[cl][kk] = ylds[e];
          bi[cl][kk] = ylds[e + 64];
        } else {
          br[cl][kk] = yimg[e];
          bi[cl][kk] = yimg[e + 64];
        }
      }
#pragma unroll
    for (int t = 0; t < MTW; ++t) {
      const int mt = w + NW * t;
      if (mt >= f.nwy) continue;
      const int mc = 16 * mt + m;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int sl = 4 * g + i;
        const float2 va = vlds[sl * f.mrow + mc];
        float2 xs[NCY];
        if constexpr (NCY == 2) {
          const float2 vbv = vlds[(16 + sl) * f.mrow + mc];
          xs[0] = make_float2(va.x + vbv.x, va.y + vbv.y);
          xs[1] = make_float2(va.x - vbv.x, va.y - vbv.y);
        } else {
          xs[0] = va;
        }
#pragma unroll
        for (int cl = 0; cl < NCY; ++cl)
#pragma unroll
          for (int kk = 0; kk < KYT; ++kk) {
            yr[cl][kk][t] = mfma(br[cl][kk][i], xs[cl].x, yr[cl][kk][t]);
            yi[cl][kk][t] = mfma(br[cl][kk][i], xs[cl].y, yi[cl][kk][t]);
            yr[cl][kk][t] = mfma(bi[cl][kk][i], -xs[cl].y, yr[cl][kk][t]);
            yi[cl][kk][t] = mfma(bi[cl][kk][i], xs[cl].x, yi[cl][kk][t]);
          }
      }
      if (c.q == f.jq - 1) {
        // Plane done: rows p of K_y (class cl, slot 16kk + 4g + i), columns mc.
        float2* op = out + c.pl * int64_t(f.ky) * f.mcols;
#pragma unroll
        for (int cl = 0; cl < NCY; ++cl)
#pragma unroll
          for (int kk = 0; kk < KYT; ++kk) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int sl = 16 * kk + 4 * g + i;
              const int p = NCY == 2 ? 2 * sl + cl : sl;
              if (p < f.ky && mc < f.mcols)
                op[int64_t(p) * f.mcols + mc] = make_float2(yr[cl][kk][t][i], yi[cl][kk][t][i]);
            }
            yr[cl][kk][t] = v4f{0.f, 0.f, 0.f, 0.f};
            yi[cl][kk][t] = v4f{0.f, 0.f, 0.f, 0.f};
          }
      }
    }
    __syncthreads();
  };

  // Tiles in order through buffers 0, 1, ..., NB - 1, 0, ...; every pass runs
  // all NB steps (steps past the last plane only load), and the only exit is
  // at the end of a pass.  The buffer index is a compile-time constant at
  // every step (the buffers stay in registers), and no path leaves a step
  // early: an exit between steps would give the compiler a path on which a
  // buffer's loads are followed by fewer loads than the other buffers', and
  // its waits for that buffer would then cover all outstanding loads.
  static_assert(NB >= 1 && NB <= 4, "one to four tile buffers");
  auto step = [&](auto kc) __attribute__((always_inline)) {
    constexpr int k = decltype(kc)::value;
    process(k);
  };
  do {
    step(std::integral_constant<int, 0>{});
    if constexpr (NB > 1) step(std::integral_constant<int, 1>{});
    if constexpr (NB > 2) step(std::integral_constant<int, 2>{});
    if constexpr (NB > 3) step(std::integral_constant<int, 3>{});
  } while (cb[0].pl < f.planes);
}

// Register budget: the common shapes fit 4 waves per SIMD (128 registers);
// the t-folded forward up to 16 accumulator tiles fits 2 (256 registers);
// the widest ones (many z classes / k_t tiles) are left to the compiler.
#define DTST_STREAM_WAVES(CT, MT, NCLS, TH, TWO) \
  __attribute__((amdgpu_waves_per_eu(((CT) * (MT) * (NCLS) <= 4 && (TH) <= 2)   ? 4 \
                                     : ((TWO) && (CT) * (MT) * (NCLS) <= 16) ? 2 \
                                                                             : 1)))

template <int CT, int TH, int MT, int NCLS, int MODE, int TF>
__global__ void __launch_bounds__(256) DTST_STREAM_WAVES(CT, MT, NCLS, TH, TF)
fwd_tz_kernel(const float* __restrict__ x, float2* __restrict__ out,
              const float* __restrict__ timg, const float4* __restrict__ zimg, StreamArgs a) {
  extern __shared__ float4 lds[];
  const int nimg = NCLS * a.zt * (TF ? 3 * MT / 2 : MT) * 64;  // image blocks per (class, z tile)
  for (int i = threadIdx.x; i < nimg; i += blockDim.x) lds[i] = zimg[i];
  __syncthreads();

  const int lane = threadIdx.x & 63;
  // B operand of the t contraction, step s = 4h + j covers t = 16h + 4g + j
  // (with TF only the first half: the folded t < N_t/2).
  float bt[TH * 4][CT];
#pragma unroll
  for (int s = 0; s < TH * 4; ++s)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) bt[s][ct] = (TF && s >= TH * 2) ? 0.f : timg[(s * CT + ct) * 64 + lane];

  const int wpb = blockDim.x >> 6;
  const int64_t wstride = int64_t(gridDim.x) * wpb;
  const int64_t wave = int64_t(blockIdx.x) * wpb + (threadIdx.x >> 6);
  if (wave >= a.rows) return;
  fwd_tz_body<CT, TH, MT, NCLS, MODE, TF>(x, out, bt, lds, a, wave, wstride);
}

// ---------------------------------------------------------------------------
// Inverse: in (rows x K_z x K_t) complex -> y (rows x N_z x N_t) fp32.
//
// load_u fetches the spectrum values of one row that this lane needs,
// build_a arranges them as the A operand of the z expansion, and inv_row runs,
// per z-tile, the z expansion (one accumulator chain per class and column
// tile), the unfold, and the t expansion (one chain per output tile) as
// interleaved MFMA phases, with all stores of the tile after them.
// MODE 0: scalar stores (N_t % 4 != 0); 1: 16-byte stores with masks;
// 2: 16-byte stores of complete tiles, no masks.
// ---------------------------------------------------------------------------

template <int CT, int TH, int MT, int NCLS, int MODE, int TF = 0>
__device__ __forceinline__ void inv_row(const float (&A)[NCLS][CT][MT][4], float* __restrict__ yrow,
                                        const float (&ta)[TH][CT][4], const float4* lds, const StreamArgs& a,
                                        int lane) {
  const int m = lane & 15, g = lane >> 4;
  for (int zt = 0; zt < a.zt; ++zt) {
    float4 B[NCLS][MT];
#pragma unroll
    for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
      for (int q = 0; q < MT; ++q) B[cl][q] = lds[((cl * a.zt + zt) * MT + q) * 64 + lane];

    v4f W[NCLS][CT];
#pragma unroll
    for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
      for (int ct = 0; ct < CT; ++ct) W[cl][ct] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < MT; ++q)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) W[cl][ct] = mfma(A[cl][ct][q][i], B[cl][q][i], W[cl][ct]);
    unfold_classes<NCLS, CT, TF>(W);
    // The t expansion and the stores run over groups of HG output z classes
    // (all of them at once, except the four-class fold of one row tile, whose
    // sixteen-wave inverse keeps two groups of two within its registers).
    constexpr int HG = (NCLS == 4 && MT == 1) ? 1 : NCLS;
    const int zl = zt * 16 + m;
    const bool zok = zl < a.zh;
#pragma unroll
    for (int h0 = 0; h0 < NCLS; h0 += HG) {
      v4f Y[HG][TH];
#pragma unroll
      for (int hh = 0; hh < HG; ++hh)
#pragma unroll
        for (int mt = 0; mt < TH; ++mt) Y[hh][mt] = v4f{0.f, 0.f, 0.f, 0.f};
      if constexpr (TF) {
        // Even k_t (tile 0) into Y[.][mt], odd k_t (tile 1) into
        // Y[.][mt + TH/2], for t < N_t/2; then E + O at t, E - O at t + N_t/2.
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int hh = 0; hh < HG; ++hh)
#pragma unroll
            for (int mt = 0; mt < TH / 2; ++mt) {
              Y[hh][mt] = mfma(ta[mt][0][i], W[h0 + hh][0][i], Y[hh][mt]);
              Y[hh][mt + TH / 2] = mfma(ta[mt][1][i], W[h0 + hh][1][i], Y[hh][mt + TH / 2]);
            }
#pragma unroll
        for (int hh = 0; hh < HG; ++hh)
#pragma unroll
          for (int mt = 0; mt < TH / 2; ++mt) {
            const v4f e = Y[hh][mt], o = Y[hh][mt + TH / 2];
            Y[hh][mt] = e + o;
            Y[hh][mt + TH / 2] = e - o;
          }
      } else {
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int hh = 0; hh < HG; ++hh)
#pragma unroll
              for (int mt = 0; mt < TH; ++mt) Y[hh][mt] = mfma(ta[mt][ct][i], W[h0 + hh][ct][i], Y[hh][mt]);
      }

      if (MODE != 0 && TH == 2 && a.nt == 32) {
        // Rows of exactly 32 floats: lanes m and m^8 trade one 16-byte
        // chunk (DPP row rotate by 8) so that each store instruction writes
        // 8 whole 128-byte rows instead of 16 half rows.
        const bool lo = m < 8;
        const int za = zt * 16 + (m & 7), zb = za + 8;
        const int tch = (lo ? 0 : 16) + 4 * g;
#pragma unroll
        for (int hh = 0; hh < HG; ++hh) {
          const int hf = h0 + hh;
          float va[4], vb[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            // lanes m >= 8 take the first tile of lane m - 8, lanes m < 8
            // the second tile of lane m + 8 (bank-masked DPP moves)
            va[i] = ror8_into<0xC>(Y[hh][0][i], Y[hh][TH - 1][i]);
            vb[i] = ror8_into<0x3>(Y[hh][TH - 1][i], Y[hh][0][i]);
          }
          if (MODE == 2 || za < a.zh)
            store_stream(yrow + int64_t(za + hf * a.zh) * a.nt + tch, va[0], va[1], va[2], va[3]);
          if (MODE == 2 || zb < a.zh)
            store_stream(yrow + int64_t(zb + hf * a.zh) * a.nt + tch, vb[0], vb[1], vb[2], vb[3]);
        }
        continue;
      }
#pragma unroll
      for (int hh = 0; hh < HG; ++hh) {
        float* dst = yrow + int64_t(zl + (h0 + hh) * a.zh) * a.nt;
#pragma unroll
        for (int mt = 0; mt < TH; ++mt) {
          const int t0 = 16 * mt + 4 * g;
          if (MODE != 0) {
            if (MODE == 2 || (zok && t0 < a.nt))
              store_stream(dst + t0, Y[hh][mt][0], Y[hh][mt][1], Y[hh][mt][2], Y[hh][mt][3]);
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (zok && t0 + i < a.nt) __builtin_nontemporal_store(Y[hh][mt][i], dst + t0 + i);
          }
        }
      }
    }
  }
}


// The A operands of the three products, Ur + Ui, Ur and Ui, are formed from
// the lane's spectrum values per z tile (zero where the mode or k_t is not
// retained), so that u is the only per-row state.
template <int TH, int MT, int NCLS, int MODE>
__device__ __forceinline__ void inv_row_tfg(const float2 (&u)[NCLS][MT / 2][4], float* __restrict__ yrow,
                                            const float (&ta)[TH][2][4], const float4* lds, const StreamArgs& a,
                                            int lane) {
  static_assert(TH % 2 == 0 && MODE != 0, "t folding needs whole 16-byte t groups");
  const int m = lane & 15, g = lane >> 4;
  constexpr int MTI = 3 * MT / 2;  // image blocks per (class, z tile)
  // the row's A operands Ur + Ui, Ur, Ui (zero where the mode or k_t is not
  // retained), formed once for every z tile
  float us[NCLS][MT / 2][4], ur[NCLS][MT / 2][4], ui[NCLS][MT / 2][4];
#pragma unroll
  for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
    for (int qh = 0; qh < MT / 2; ++qh)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool ok = tfg_index<NCLS>(a, m, g, cl, qh, i) >= 0;
        ur[cl][qh][i] = ok ? u[cl][qh][i].x : 0.f;
        ui[cl][qh][i] = ok ? u[cl][qh][i].y : 0.f;
        us[cl][qh][i] = ur[cl][qh][i] + ui[cl][qh][i];
      }
  for (int zt = 0; zt < a.zt; ++zt) {
    v4f Wr[NCLS], Wi[NCLS];
#pragma unroll
    for (int cl = 0; cl < NCLS; ++cl) {
      v4f k1 = v4f{0.f, 0.f, 0.f, 0.f}, k2 = k1, k3 = k1;
#pragma unroll
      for (int qh = 0; qh < MT / 2; ++qh) {
        // z image blocks of these K entries: Cr, Ci - Cr, Cr + Ci (C_z = Cr + i Ci)
        const float4* zb = lds + ((cl * a.zt + zt) * MTI + qh) * 64 + lane;
        const float4 cr = zb[0], dm = zb[(MT / 2) * 64], sp = zb[MT * 64];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          k1 = mfma(us[cl][qh][i], cr[i], k1);
          k2 = mfma(ur[cl][qh][i], dm[i], k2);
          k3 = mfma(ui[cl][qh][i], sp[i], k3);
        }
      }
      Wr[cl] = k1 - k3;
      Wi[cl] = k1 + k2;
    }
    if constexpr (NCLS == 2) {
      // even modes + odd modes at z, even - odd at z + N_z/2
      const v4f sr = Wr[0] + Wr[1], dr = Wr[0] - Wr[1];
      const v4f si = Wi[0] + Wi[1], di = Wi[0] - Wi[1];
      Wr[0] = sr;
      Wr[1] = dr;
      Wi[0] = si;
      Wi[1] = di;
    } else if constexpr (NCLS == 4) {
      // y0 = (E0 + E2) + (E1 + E3)      y2 = (E0 + E2) - (E1 + E3)
      // y1 = (E0 - E2) + i (E1 - E3)    y3 = (E0 - E2) - i (E1 - E3)
      const v4f ar = Wr[0] + Wr[2], ai = Wi[0] + Wi[2];
      const v4f br = Wr[1] + Wr[3], bi = Wi[1] + Wi[3];
      const v4f cr = Wr[0] - Wr[2], ci = Wi[0] - Wi[2];
      const v4f dr = Wr[1] - Wr[3], di = Wi[1] - Wi[3];
      Wr[0] = ar + br;
      Wi[0] = ai + bi;
      Wr[2] = ar - br;
      Wi[2] = ai - bi;
      Wr[1] = cr - di;  // c + i d
      Wi[1] = ci + dr;
      Wr[3] = cr + di;  // c - i d
      Wi[3] = ci - dr;
    }
    const int zl = zt * 16 + m;
#pragma unroll
    for (int hf = 0; hf < NCLS; ++hf) {
      // even k_t (registers 0, 1) into E, odd (2, 3) into O, for t < N_t/2
      v4f E[TH / 2], O[TH / 2];
#pragma unroll
      for (int mt = 0; mt < TH / 2; ++mt) {
        E[mt] = v4f{0.f, 0.f, 0.f, 0.f};
        O[mt] = v4f{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int mt = 0; mt < TH / 2; ++mt) {
          v4f& acc = i < 2 ? E[mt] : O[mt];
          acc = mfma(ta[mt][0][i], Wr[hf][i], acc);
          acc = mfma(ta[mt][1][i], Wi[hf][i], acc);
        }
      v4f Y[TH];
#pragma unroll
      for (int mt = 0; mt < TH / 2; ++mt) {
        Y[mt] = E[mt] + O[mt];
        Y[mt + TH / 2] = E[mt] - O[mt];
      }
      if (TH == 2 && a.nt == 32) {
        // lanes m and m^8 trade one 16-byte chunk so that each store writes
        // 8 whole 128-byte rows
        const bool lo = m < 8;
        const int za = zt * 16 + (m & 7), zb = za + 8;
        const int tch = (lo ? 0 : 16) + 4 * g;
        float va[4], vb[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          va[i] = ror8_into<0xC>(Y[0][i], Y[TH - 1][i]);
          vb[i] = ror8_into<0x3>(Y[TH - 1][i], Y[0][i]);
        }
        if (MODE == 2 || za < a.zh)
          store_stream(yrow + int64_t(za + hf * a.zh) * a.nt + tch, va[0], va[1], va[2], va[3]);
        if (MODE == 2 || zb < a.zh)
          store_stream(yrow + int64_t(zb + hf * a.zh) * a.nt + tch, vb[0], vb[1], vb[2], vb[3]);
      } else {
        float* dst = yrow + int64_t(zl + hf * a.zh) * a.nt;
#pragma unroll
        for (int mt = 0; mt < TH; ++mt) {
          const int t0 = 16 * mt + 4 * g;
          if (MODE == 2 || (zl < a.zh && t0 < a.nt))
            store_stream(dst + t0, Y[mt][0], Y[mt][1], Y[mt][2], Y[mt][3]);
        }
      }
    }
  }
}

// Each row's spectrum is loaded one row ahead (except in the t-folded
// instances, see below).
template <int CT, int TH, int MT, int NCLS, int MODE, int TF>
__device__ __forceinline__ void inv_zt_body(const float2* __restrict__ in, float* __restrict__ y,
                                            const float (&ta)[TH][CT][4], const float4* lds,
                                            const StreamArgs& a, int64_t wave, int64_t wstride) {
  const int lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int64_t row_len = int64_t(a.nz) * a.nt;
  const int64_t spec_len = int64_t(a.kz) * a.kt;

  if constexpr (TF) {
    // Two spectrum buffers: while one row is expanded the next row's values
    // are in flight in the other; passes of two rows keep the buffer index a
    // compile-time constant, and the loads are unconditional (past the last
    // row the wave re-reads its last row, which is not expanded again).
    const int64_t n_rows = (a.rows - 1 - wave) / wstride + 1;
    const int64_t last_row = wave + (n_rows - 1) * wstride;
    float2 ub[2][NCLS][MT / 2][4];
    int64_t rp[2];
    int64_t rn = wave;
    auto fetch = [&](int k) __attribute__((always_inline)) {
      rp[k] = rn;
      load_u_tfg<MT, NCLS>(in + (rn < last_row ? rn : last_row) * spec_len, a, m, g, ub[k]);
      rn += wstride;
    };
    fetch(0);
    fetch(1);
    auto step = [&](auto kc) __attribute__((always_inline)) {
      constexpr int k = decltype(kc)::value;
      const int64_t r = rp[k];
      if (r <= last_row) inv_row_tfg<TH, MT, NCLS, MODE>(ub[k], y + r * row_len, ta, lds, a, lane);
      fetch(k);
    };
    do {
      step(std::integral_constant<int, 0>{});
      step(std::integral_constant<int, 1>{});
    } while (rp[0] <= last_row);
    return;
  }
  float2 un[NCLS][CT][USlots<MT>::QH][4];
  load_u<CT, MT, NCLS, TF>(in + wave * spec_len, a, m, g, un);
  for (int64_t r = wave; r < a.rows; r += wstride) {
    float A[NCLS][CT][MT][4];
    build_a<CT, MT, NCLS, TF>(un, a, m, g, A);
    if (r + wstride < a.rows) load_u<CT, MT, NCLS, TF>(in + (r + wstride) * spec_len, a, m, g, un);
    inv_row<CT, TH, MT, NCLS, MODE, TF>(A, y + r * row_len, ta, lds, a, lane);
  }
}

template <int CT, int TH, int MT, int NCLS, int MODE, int TF>
__global__ void __launch_bounds__(256) DTST_STREAM_WAVES(CT, MT, NCLS, TH, TF)
inv_zt_kernel(const float2* __restrict__ in, float* __restrict__ y,
              const float* __restrict__ timg, const float4* __restrict__ zimg, StreamArgs a) {
  extern __shared__ float4 lds[];
  const int nimg = NCLS * a.zt * (TF ? 3 * MT / 2 : MT) * 64;  // image blocks per (class, z tile)
  for (int i = threadIdx.x; i < nimg; i += blockDim.x) lds[i] = zimg[i];
  __syncthreads();

  const int lane = threadIdx.x & 63;
  // A operand of the t expansion: rows t = 16mt + m, K index c = 16ct + 4g + i
  // (with TF only mt < TH/2: the folded t < N_t/2).
  float ta[TH][CT][4];
#pragma unroll
  for (int mt = 0; mt < TH; ++mt)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        ta[mt][ct][i] = (TF && mt >= TH / 2) ? 0.f : timg[((mt * CT + ct) * 4 + i) * 64 + lane];

  const int wpb = blockDim.x >> 6;
  const int64_t wstride = int64_t(gridDim.x) * wpb;
  const int64_t wave = int64_t(blockIdx.x) * wpb + (threadIdx.x >> 6);
  if (wave >= a.rows) return;
  inv_zt_body<CT, TH, MT, NCLS, MODE, TF>(in, y, ta, lds, a, wave, wstride);
}

// ---------------------------------------------------------------------------
// Inverse y + z + t in one pass (same shape conditions as fwd_tzy_kernel).
//
// A workgroup of 16 waves owns one (b, c, x) plane (one workgroup per plane:
// a persistent loop would make every plane's operand loads wait behind the
// previous plane's outstanding row stores, which share the wave's memory
// counter).  Wave w < ceil(K_z K_t / 16) loads the columns 16w..16w+15 of the
// plane's (K_y x K_z K_t) spectrum as MFMA B operands (K index = y mode).  For
// every group of 16 slots (one y tile of the inverse y image) those waves
// expand y for the group's slots -- folded, the even-mode sum E and odd-mode
// sum O give E + O at y and E - O at y + N_y/2 -- and leave the rows in LDS;
// after a barrier, wave w expands z and t of the row(s) of slot w exactly as
// inv_zt_body does and streams them out; a second barrier frees the LDS rows.
// The (N_y x K_z K_t) intermediate never reaches HBM.
// ---------------------------------------------------------------------------
template <int TH, int NCLS, int MODE, int NCY, int JQY, int YL>
__global__ void __launch_bounds__(1024)
inv_yzt_kernel(const float2* __restrict__ in, float* __restrict__ y, const float* __restrict__ timg,
               const float4* __restrict__ zimg, const float4* __restrict__ yimg, StreamArgs a, FusedArgs f) {
  constexpr int CT = 1, MT = NCLS == 4 ? 1 : 2;
  extern __shared__ float4 lds[];
  const int nimg = NCLS * a.zt * MT * 64;
  float2* vlds = reinterpret_cast<float2*>(lds + nimg);
  const int lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int w = threadIdx.x >> 6;
  if (blockIdx.x >= f.planes) return;  // the host launches one workgroup per plane
  const int64_t pl = blockIdx.x;
  const int mc = 16 * w + m;
  const bool col_ok = mc < f.mcols;

  // LDS: z image, the exchanged rows, the y image (YL = 1; with YL = 0 the
  // y image is read from global memory).  The staging loads go out first,
  // then the spectrum operands and the t basis, which stay in flight across
  // the staging barrier.
  float4* ylds = reinterpret_cast<float4*>(vlds + 16 * NCY * f.mrow);
  const StageLast stl = stage_begin(lds, zimg, yimg, nimg, YL ? f.yimg_n4 : 0, 8 * NCY * f.mrow);

  // B operands of the y expansion: spectrum row p (class cl, K index
  // 16q + 4g + i), column mc.  The loads are unconditional (lanes outside the
  // spectrum read its first value) and u_ok masks them where they are used:
  // a load under a condition would make the staging stores below wait for
  // every outstanding load.
  auto u_ok = [&](int cl, int q, int i) {
    const int kk = 16 * q + 4 * g + i;
    const int p = NCY == 2 ? 2 * kk + cl : kk;
    return col_ok && p < f.ky;
  };
  float2 u[NCY][JQY][4];
  {
    const float2* sp = in + pl * int64_t(f.ky) * f.mcols;
#pragma unroll
    for (int cl = 0; cl < NCY; ++cl)
#pragma unroll
      for (int q = 0; q < JQY; ++q)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int kk = 16 * q + 4 * g + i;
          const int p = NCY == 2 ? 2 * kk + cl : kk;
          u[cl][q][i] = sp[u_ok(cl, q, i) ? int64_t(p) * f.mcols + mc : 0];
        }
  }

  // A operand of the t expansion: rows t = 16mt + m, K index c = 4g + i.
  float ta[TH][CT][4];
#pragma unroll
  for (int mt = 0; mt < TH; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) ta[mt][0][i] = timg[(mt * 4 + i) * 64 + lane];
  // y image from global memory (YL = 0): the entries of group gq are held in
  // registers, and those of the next group are loaded right after the
  // group's y expansion, before its row stores: read at the group start they
  // would wait for the previous group's stores (one memory counter per wave)
  float4 yb[YL ? 1 : JQY][YL ? 1 : NCY][2];
  auto load_y = [&](int gq) __attribute__((always_inline)) {
    if constexpr (!YL) {
#pragma unroll
      for (int q = 0; q < JQY; ++q)
#pragma unroll
        for (int cl = 0; cl < NCY; ++cl) {
          const int e = ((gq * JQY + q) * NCY + cl) * 2 * 64 + lane;
          yb[q][cl][0] = yimg[e];
          yb[q][cl][1] = yimg[e + 64];
        }
    }
  };
  load_y(0);
  stage_end(lds, stl);
  __syncthreads();

  const int64_t row_len = int64_t(a.nz) * a.nt;
  {
    for (int gq = 0; gq < f.jq; ++gq) {
      if (w < f.nwy) {
        v4f er[NCY], ei[NCY];
#pragma unroll
        for (int cl = 0; cl < NCY; ++cl) {
          er[cl] = v4f{0.f, 0.f, 0.f, 0.f};
          ei[cl] = v4f{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int q = 0; q < JQY; ++q)
#pragma unroll
          for (int cl = 0; cl < NCY; ++cl) {
            // image entry (((tile * JQ + q) * NCY + class) * 2 + part) * 64 + lane
            const int e = ((gq * JQY + q) * NCY + cl) * 2 * 64 + lane;
            const float4 br = YL ? ylds[e] : yb[YL ? 0 : q][YL ? 0 : cl][0];
            const float4 bi = YL ? ylds[e + 64] : yb[YL ? 0 : q][YL ? 0 : cl][1];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float2 v = u_ok(cl, q, i) ? u[cl][q][i] : make_float2(0.f, 0.f);
              er[cl] = mfma(br[i], v.x, er[cl]);
              ei[cl] = mfma(br[i], v.y, ei[cl]);
              er[cl] = mfma(bi[i], -v.y, er[cl]);
              ei[cl] = mfma(bi[i], v.x, ei[cl]);
            }
          }
        // accumulator register i holds slot 4g + i, column mc
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int sl = 4 * g + i;
          if constexpr (NCY == 2) {
            vlds[sl * f.mrow + mc] = make_float2(er[0][i] + er[1][i], ei[0][i] + ei[1][i]);
            vlds[(16 + sl) * f.mrow + mc] = make_float2(er[0][i] - er[1][i], ei[0][i] - ei[1][i]);
          } else {
            vlds[sl * f.mrow + mc] = make_float2(er[0][i], ei[0][i]);
          }
        }
      }
      load_y(gq + 1 < f.jq ? gq + 1 : gq);
      __syncthreads();
      const int s = 16 * gq + w;
      if (s < f.slots) {
#pragma unroll
        for (int h = 0; h < NCY; ++h) {
          float2 uu[NCLS][CT][USlots<MT>::QH][4];
          load_u<CT, MT, NCLS>(vlds + (h * 16 + w) * f.mrow, a, m, g, uu);
          float A[NCLS][CT][MT][4];
          build_a<CT, MT, NCLS>(uu, a, m, g, A);
          inv_row<CT, TH, MT, NCLS, MODE>(A, y + (pl * f.ny + s + h * f.half) * row_len, ta, lds, a, lane);
        }
      }
      __syncthreads();
    }
  }
}

typedef void (*fwd_fn)(const float*, float2*, const float*, const float4*, StreamArgs);
typedef void (*ifused_fn)(const float2*, float*, const float*, const float4*, const float4*, StreamArgs, FusedArgs);
typedef void (*fused_fn)(const float*, float2*, const float*, const float4*, const float4*, StreamArgs, FusedArgs);
typedef void (*inv_fn)(const float2*, float*, const float*, const float4*, StreamArgs);

// Load / store form of a configuration: 0 scalar (N_t % 4 != 0), 1 16-byte
// with masks, 2 complete tiles (z tiles and t groups all full).  Each form is
// its own kernel instance, so the registers of one do not limit the others.
int mode_of(const StreamCfg& c) {
  if (!c.vec) return 0;
  return (c.zh % 16 == 0 && c.nt == 16 * c.th) ? 2 : 1;
}

template <int CT, int TH, int MT, int NCLS, int TF>
void pick3(int mode, fwd_fn* f, inv_fn* v) {
  if (mode == 2) {
    *f = fwd_tz_kernel<CT, TH, MT, NCLS, 2, TF>;
    *v = inv_zt_kernel<CT, TH, MT, NCLS, 2, TF>;
  } else if (mode == 1) {
    *f = fwd_tz_kernel<CT, TH, MT, NCLS, 1, TF>;
    *v = inv_zt_kernel<CT, TH, MT, NCLS, 1, TF>;
  } else if constexpr (!TF) {
    *f = fwd_tz_kernel<CT, TH, MT, NCLS, 0, TF>;
    *v = inv_zt_kernel<CT, TH, MT, NCLS, 0, TF>;
  } else {
    *f = nullptr;  // no scalar-load form of the t-folded kernels
    *v = nullptr;
  }
}

template <int CT, int TH, int MT, int TF>
void pick2(int ncls, int mode, fwd_fn* f, inv_fn* v) {
  if constexpr (MT == 1) {
    // one row tile per class: the four-class fold of one column tile only
    if (ncls == 4) {
      pick3<CT, TH, 1, 4, TF>(mode, f, v);
    } else {
      *f = nullptr;
      *v = nullptr;
    }
  } else {
    if constexpr (CT == 2 && MT == 2) {
      if (ncls == 4) {
        pick3<CT, TH, MT, 4, TF>(mode, f, v);
        return;
      }
    }
    if (ncls == 2) pick3<CT, TH, MT, 2, TF>(mode, f, v);
    else pick3<CT, TH, MT, 1, TF>(mode, f, v);
  }
}

template <int CT, int TH, int TF>
void pick1(int mt, int ncls, int mode, fwd_fn* f, inv_fn* v) {
  if constexpr (CT == 1 && !TF) {
    if (mt == 1) {
      pick2<CT, TH, 1, TF>(ncls, mode, f, v);
      return;
    }
  }
  if (mt == 2) pick2<CT, TH, 2, TF>(ncls, mode, f, v);
  else if (mt == 4) pick2<CT, TH, 4, TF>(ncls, mode, f, v);
  else pick2<CT, TH, 8, TF>(ncls, mode, f, v);
}

template <int CT>
void pick0(int th, int mt, int ncls, int mode, fwd_fn* f, inv_fn* v) {
  if (th == 1) pick1<CT, 1, 0>(mt, ncls, mode, f, v);
  else if (th == 2) pick1<CT, 2, 0>(mt, ncls, mode, f, v);
  else pick1<CT, 4, 0>(mt, ncls, mode, f, v);
}

template <int TH, int NCLS, int MODE, int YL>
fused_fn pick_fused4(int ncy, int kyt) {
  constexpr int NB = NCLS == 4 ? kFusedBufs4 : kFusedBufs;
  if (ncy == 2) return fwd_tzy_kernel<TH, NCLS, MODE, 2, 1, kFusedWaves, NB, YL>;
  if (kyt == 1) return fwd_tzy_kernel<TH, NCLS, MODE, 1, 1, kFusedWaves, NB, YL>;
  return fwd_tzy_kernel<TH, NCLS, MODE, 1, 2, kFusedWaves, NB, YL>;
}

template <int TH, int NCLS, int MODE>
fused_fn pick_fused3(int ncy, int kyt, int yl) {
  return yl ? pick_fused4<TH, NCLS, MODE, 1>(ncy, kyt) : pick_fused4<TH, NCLS, MODE, 0>(ncy, kyt);
}

template <int TH, int NCLS>
fused_fn pick_fused2(int mode, int ncy, int kyt, int yl) {
  return mode == 2 ? pick_fused3<TH, NCLS, 2>(ncy, kyt, yl) : pick_fused3<TH, NCLS, 1>(ncy, kyt, yl);
}

template <int TH, int NCLS, int MODE, int YL>
ifused_fn pick_ifused4(int ncy, int jqy) {
  if (ncy == 2) return inv_yzt_kernel<TH, NCLS, MODE, 2, 1, YL>;
  if (jqy == 1) return inv_yzt_kernel<TH, NCLS, MODE, 1, 1, YL>;
  return inv_yzt_kernel<TH, NCLS, MODE, 1, 2, YL>;
}

template <int TH, int NCLS, int MODE>
ifused_fn pick_ifused3(int ncy, int jqy, int yl) {
  return yl ? pick_ifused4<TH, NCLS, MODE, 1>(ncy, jqy) : pick_ifused4<TH, NCLS, MODE, 0>(ncy, jqy);
}

template <int TH, int NCLS>
ifused_fn pick_ifused2(int mode, int ncy, int jqy, int yl) {
  return mode == 2 ? pick_ifused3<TH, NCLS, 2>(ncy, jqy, yl) : pick_ifused3<TH, NCLS, 1>(ncy, jqy, yl);
}

// Fused y + z + t instances: as below, with JQY 16-wide K steps per y class
// and the y image in LDS (YL = 1) or read from global memory.
ifused_fn pick_ifused(const StreamCfg& c) {
  const int mode = mode_of(c), yl = c.fused_y_lds;
  if (c.th == 1) {
    if (c.ncls == 4) return pick_ifused2<1, 4>(mode, c.ncy, c.kyt, yl);
    return c.ncls == 2 ? pick_ifused2<1, 2>(mode, c.ncy, c.kyt, yl) : pick_ifused2<1, 1>(mode, c.ncy, c.kyt, yl);
  }
  if (c.ncls == 4) return pick_ifused2<2, 4>(mode, c.ncy, c.kyt, yl);
  return c.ncls == 2 ? pick_ifused2<2, 2>(mode, c.ncy, c.kyt, yl) : pick_ifused2<2, 1>(mode, c.ncy, c.kyt, yl);
}

// Fused t + z + y instances: CT = 1, TH <= 2, 16-byte loads, NCLS <= 2 with
// MT = 2 or NCLS = 4 with MT = 1; (NCY, KYT) = (2, 1) folded, (1, 1) or
// (1, 2) otherwise.
fused_fn pick_fused(const StreamCfg& c) {
  const int mode = mode_of(c), yl = c.fused_y_lds;
  if (c.th == 1) {
    if (c.ncls == 4) return pick_fused2<1, 4>(mode, c.ncy, c.kyt, yl);
    return c.ncls == 2 ? pick_fused2<1, 2>(mode, c.ncy, c.kyt, yl) : pick_fused2<1, 1>(mode, c.ncy, c.kyt, yl);
  }
  if (c.ncls == 4) return pick_fused2<2, 4>(mode, c.ncy, c.kyt, yl);
  return c.ncls == 2 ? pick_fused2<2, 2>(mode, c.ncy, c.kyt, yl) : pick_fused2<2, 1>(mode, c.ncy, c.kyt, yl);
}

// Split t + z and z + t instances; the t-folded ones (tf: CT = 2, N_t = 32,
// 16-byte loads) are their own set.
void pick(const StreamCfg& c, fwd_fn* f, inv_fn* v) {
  if (c.tf) pick1<2, 2, 1>(c.mt, c.ncls, mode_of(c), f, v);
  else if (c.ct == 1) pick0<1>(c.th, c.mt, c.ncls, mode_of(c), f, v);
  else pick0<2>(c.th, c.mt, c.ncls, mode_of(c), f, v);
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
  a.full = mode_of(c) == 2 ? 1 : 0;
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
  if (f == nullptr || v == nullptr) return hipErrorInvalidConfiguration;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(f),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(c->lds_bytes));
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(v), hipFuncAttributeMaxDynamicSharedMemorySize,
                          int(c->lds_bytes));
  if (e != hipSuccess) return e;
  if (c->fuse_y) {
    const void* ff = reinterpret_cast<const void*>(pick_fused(*c));
    e = hipFuncSetAttribute(ff, hipFuncAttributeMaxDynamicSharedMemorySize, int(c->fused_lds_bytes));
    if (e != hipSuccess) return e;
    int dev = 0, cus = 0, per_cu = 0;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, ff, 64 * kFusedWaves, c->fused_lds_bytes)) !=
        hipSuccess)
      return e;
    c->grid_fused = cus * (per_cu > 0 ? per_cu : 1);
    const void* fi = reinterpret_cast<const void*>(pick_ifused(*c));
    e = hipFuncSetAttribute(fi, hipFuncAttributeMaxDynamicSharedMemorySize, int(c->fused_lds_bytes));
    if (e != hipSuccess) return e;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fi, 1024, c->fused_lds_bytes)) != hipSuccess)
      return e;
    if (per_cu <= 0) return hipErrorInvalidConfiguration;
  }
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

int launch_fwd_tzy(const StreamCfg& c, const AxisCfg& ay, const float* x, void* out, int64_t planes, int ny,
                   const float* timg, const float* zimg, const float* yimg, void* stream) {
  if (planes <= 0) return hipSuccess;
  FusedArgs f;
  f.planes = planes;
  f.ny = ny;
  f.slots = ay.fold == 1 ? ny / 2 : ny;
  f.half = ay.fold == 1 ? ny / 2 : 0;
  f.jq = ay.JQ;
  f.kth = ay.kth;
  f.ky = ay.KO;
  f.mcols = c.kz * c.kt;
  f.mrow = c.fused_mrow;
  f.nwy = (f.mcols + 15) / 16;
  f.yimg_n4 = ay.ktiles * ay.JQ * 2 * 64;
  const int64_t grid = planes < c.grid_fused ? planes : c.grid_fused;
  hipLaunchKernelGGL(pick_fused(c), dim3(static_cast<unsigned>(grid)), dim3(64 * kFusedWaves), c.fused_lds_bytes,
                     static_cast<hipStream_t>(stream), x, static_cast<float2*>(out), timg,
                     reinterpret_cast<const float4*>(zimg), reinterpret_cast<const float4*>(yimg),
                     args_of(c, planes * ny), f);
  return hipGetLastError();
}

int launch_inv_yzt(const StreamCfg& c, const AxisCfg& ay, const void* in, float* y, int64_t planes, int ny,
                   const float* timg, const float* zimg, const float* yimg, void* stream) {
  if (planes <= 0) return hipSuccess;
  // The y expansion's image must have the K steps and tiles the kernel assumes.
  if (ay.JQ != c.kyt || (ay.fold == 2) != (c.ncy == 2)) return hipErrorInvalidValue;
  FusedArgs f;
  f.planes = planes;
  f.ny = ny;
  f.slots = ay.fold == 2 ? ny / 2 : ny;
  f.half = ay.fold == 2 ? ny / 2 : 0;
  f.jq = ay.ktiles;
  f.kth = 0;
  f.ky = ay.J;
  f.mcols = c.kz * c.kt;
  f.mrow = c.fused_mrow;
  f.nwy = (f.mcols + 15) / 16;
  f.yimg_n4 = ay.ktiles * ay.JQ * (ay.fold == 2 ? 2 : 1) * 2 * 64;
  if (planes > int64_t(0x7fffffff)) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(pick_ifused(c), dim3(static_cast<unsigned>(planes)), dim3(1024), c.fused_lds_bytes,
                     static_cast<hipStream_t>(stream), static_cast<const float2*>(in), y, timg,
                     reinterpret_cast<const float4*>(zimg), reinterpret_cast<const float4*>(yimg),
                     args_of(c, planes * ny), f);
  return hipGetLastError();
}

}  // namespace dtst
