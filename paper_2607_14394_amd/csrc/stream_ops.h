// Device helpers shared by the streaming kernels (k_stream.hip) and the
// fused inverse + block epilogue kernel (k_block_zt.hip): the MFMA wrapper,
// lane exchanges, the z class fold / unfold, and the loads and operand
// layouts of the inverse's z expansion.  Included inside namespace
// dtst::{anonymous}; every translation unit gets its own copy.
#pragma once

typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4f mfma(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// The inverse's real output is written once and not read again by this
// library: stream it past the caches.
__device__ __forceinline__ void store_stream(float* p, float a, float b, float c, float d) {
  __builtin_nontemporal_store(v4f{a, b, c, d}, reinterpret_cast<v4f*>(p));
}

struct StreamArgs {
  int64_t rows;
  int nt, nz, kt, kz, zh, zt, vec;
  int full;  // every z tile and t group is complete: no masking needed
};

// DPP row rotate by 8 within each 16-lane row: lane m reads lane m ^ 8.
__device__ __forceinline__ float ror8(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x128, 0xf, 0xf, false));
}

// ror8 of src written only to the lanes of the DPP banks in BANKS (bank b =
// lanes 4b..4b+3 of every row of 16); the other lanes return old.
template <int BANKS>
__device__ __forceinline__ float ror8_into(float old, float src) {
  return __int_as_float(
      __builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(src), 0x128, 0xf, BANKS, false));
}

// ---------------------------------------------------------------------------
// z folding.  With z undistributed and N = N_z divisible by NCLS,
// B[k, z + jN/NCLS] = w^(kj) B[k, z] with w = -1 (NCLS = 2) or -i (NCLS = 4),
// so the modes split into NCLS classes by k mod NCLS and each class only
// needs the z < N/NCLS positions of the combination
//   S_c(z) = sum_j w^(cj) V_j(z),   V_j(z) = V(z + jN/NCLS).
// The inverse forms the class sums E_c(z) and writes
//   y(z + jN/NCLS) = sum_c conj(w)^(cj) E_c(z).
// V and E hold complex values as two column tiles (tile 0 Re, tile 1 Im) when
// CT = 2, which makes the factors +-i lane-local; NCLS = 4 is only used then.
//
// t folding (TF = 1; CT = 2, N_t = 16 TH with TH even, t undistributed).
// B_t[k, t + N_t/2] = (-1)^k B_t[k, t], so even k_t only need the sums
// x(t) + x(t + N_t/2) and odd k_t the differences, over t < N_t/2: half the
// t products.  Column tile 0 then holds the even k_t and tile 1 the odd ones.
// In the forward's t-contracted values (columns = lanes) Re of k_t = 2c + ct
// sits in lane m = c and Im in lane m = c + 8; in the inverse's z-expanded
// values (rows = accumulator registers 4g + i) k_t = 2(2g + (i & 1)) + ct
// with Re in registers 0, 1 and Im in registers 2, 3.
// ---------------------------------------------------------------------------
template <int CT>
__device__ __forceinline__ void times_i(const v4f (&a)[CT], v4f (&out)[CT]) {
  // i (re + i im) = -im + i re
  out[0] = -a[CT - 1];
  out[CT - 1] = a[0];
}

// i * a for the forward's t-folded tiles: Re and Im 8 lanes apart.
template <int CT>
__device__ __forceinline__ void times_i_lanes(const v4f (&a)[CT], v4f (&out)[CT]) {
  const float sgn = (threadIdx.x & 15) < 8 ? -1.f : 1.f;
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int i = 0; i < 4; ++i) out[ct][i] = sgn * ror8(a[ct][i]);
}

// i * a for the inverse's t-folded tiles: Re in registers 0, 1, Im in 2, 3.
template <int CT>
__device__ __forceinline__ void times_i_regs(const v4f (&a)[CT], v4f (&out)[CT]) {
#pragma unroll
  for (int ct = 0; ct < CT; ++ct) out[ct] = v4f{-a[ct][2], -a[ct][3], a[ct][0], a[ct][1]};
}

// The forward's t-contracted values hold Re and Im of k_t 8 lanes apart when
// CT = 1 (and when t folds); the inverse's z-expanded values of the four-class
// fold hold them in registers i and i + 2 of one lane (CT = 1, and t folds).
template <int NCLS, int CT, int TF = 0>
__device__ __forceinline__ void fold_classes(v4f (&V)[NCLS][CT]) {
  if constexpr (NCLS == 2) {
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      const v4f s = V[0][ct] + V[1][ct];
      const v4f d = V[0][ct] - V[1][ct];
      V[0][ct] = s;
      V[1][ct] = d;
    }
  } else if constexpr (NCLS == 4) {
    // S0 = (V0 + V2) + (V1 + V3)      S2 = (V0 + V2) - (V1 + V3)
    // S1 = (V0 - V2) - i (V1 - V3)    S3 = (V0 - V2) + i (V1 - V3)
    v4f a[CT], b[CT], c[CT], d[CT], id[CT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      a[ct] = V[0][ct] + V[2][ct];
      b[ct] = V[1][ct] + V[3][ct];
      c[ct] = V[0][ct] - V[2][ct];
      d[ct] = V[1][ct] - V[3][ct];
    }
    if constexpr (TF || CT == 1) times_i_lanes<CT>(d, id);
    else times_i<CT>(d, id);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      V[0][ct] = a[ct] + b[ct];
      V[2][ct] = a[ct] - b[ct];
      V[1][ct] = c[ct] - id[ct];
      V[3][ct] = c[ct] + id[ct];
    }
  }
}

template <int NCLS, int CT, int TF = 0>
__device__ __forceinline__ void unfold_classes(v4f (&E)[NCLS][CT]) {
  if constexpr (NCLS == 2) {
    // even modes + odd modes at z, even - odd at z + N_z/2
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      const v4f s = E[0][ct] + E[1][ct];
      const v4f d = E[0][ct] - E[1][ct];
      E[0][ct] = s;
      E[1][ct] = d;
    }
  } else if constexpr (NCLS == 4) {
    // y0 = (E0 + E2) + (E1 + E3)      y2 = (E0 + E2) - (E1 + E3)
    // y1 = (E0 - E2) + i (E1 - E3)    y3 = (E0 - E2) - i (E1 - E3)
    v4f a[CT], b[CT], c[CT], d[CT], id[CT];
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      a[ct] = E[0][ct] + E[2][ct];
      b[ct] = E[1][ct] + E[3][ct];
      c[ct] = E[0][ct] - E[2][ct];
      d[ct] = E[1][ct] - E[3][ct];
    }
    if constexpr (TF || CT == 1) times_i_regs<CT>(d, id);
    else times_i<CT>(d, id);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      E[0][ct] = a[ct] + b[ct];
      E[2][ct] = a[ct] - b[ct];
      E[1][ct] = c[ct] + id[ct];
      E[3][ct] = c[ct] - id[ct];
    }
  }
}

// k_t and part (0 Re, 1 Im) of row m of column tile ct of the inverse's z
// expansion: c = 16ct + m with c < 8CT the Re rows of k_t = c and the rest
// the Im rows of k_t = c - 8CT; with TF k_t = 2(2(m >> 2) + (m & 1)) + ct
// and part (m >> 1) & 1.
// With the four-class z fold of one column tile (CT = 1, NCLS = 4) row m is
// k_t = 2(m >> 2) + (m & 1), part (m >> 1) & 1 (Re and Im of one k_t in
// registers i and i + 2 of one lane, as with TF).
template <int CT, int TF, int NCLS = 1>
__device__ __forceinline__ void inv_row_kt(int ct, int m, int* kt, bool* is_re) {
  if constexpr (TF) {
    *kt = 2 * (2 * (m >> 2) + (m & 1)) + ct;
    *is_re = ((m >> 1) & 1) == 0;
  } else if constexpr (CT == 1 && NCLS == 4) {
    *kt = 2 * (m >> 2) + (m & 1);
    *is_re = ((m >> 1) & 1) == 0;
  } else {
    const int c = 16 * ct + m;
    *is_re = c < 8 * CT;
    *kt = *is_re ? c : c - 8 * CT;
  }
}

// Spectrum index (p * K_t + k_t) of the value this lane needs for slot
// s = 16qh + 4g + i (MT = 1: s = 2g + i, i < 2) of class cl at the k_t of
// row m of tile ct, or -1 when the mode is not retained.  A pure function of
// the lane and the shape, so the validity is recomputed where it is used
// instead of being kept in registers across the row-ahead load.
template <int CT, int NCLS, int TF, int MT = 2>
__device__ __forceinline__ int u_index(const StreamArgs& a, int m, int g, int cl, int ct, int qh, int i, bool* is_re) {
  const int s = MT == 1 ? 2 * g + i : 16 * qh + 4 * g + i;
  const int p = s * NCLS + cl;
  int kt;
  inv_row_kt<CT, TF, NCLS>(ct, m, &kt, is_re);
  return (p < a.kz && kt < a.kt) ? p * a.kt + kt : -1;
}

// Spectrum values per lane, class and column tile: 4 per pair of row tiles,
// 2 with one row tile (MT = 1).
template <int MT>
struct USlots {
  static constexpr int QH = MT == 1 ? 1 : MT / 2;
  static constexpr int N = MT == 1 ? 2 : 4;
};

// Spectrum values this lane needs from one row (Re and Im rows read the same
// value; lanes of modes that are not retained read the row start).
template <int CT, int MT, int NCLS, int TF = 0>
__device__ __forceinline__ void load_u(const float2* urow, const StreamArgs& a, int m, int g,
                                       float2 (&dst)[NCLS][CT][USlots<MT>::QH][4]) {
#pragma unroll
  for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int qh = 0; qh < USlots<MT>::QH; ++qh)
#pragma unroll
        for (int i = 0; i < USlots<MT>::N; ++i) {
          bool is_re;
          const int idx = u_index<CT, NCLS, TF, MT>(a, m, g, cl, ct, qh, i, &is_re);
          dst[cl][ct][qh][i] = urow[idx < 0 ? 0 : idx];
        }
}

// A operand of the z expansion (rows c, K index kz' = 16q + 4g + i):
// kz' < KCP pairs with Re C_z, kz' >= KCP with Im C_z; with MT = 1 K index
// 4g + i is slot 2g + (i >> 1), Re C_z for even i and Im C_z for odd i.
template <int CT, int MT, int NCLS, int TF = 0>
__device__ __forceinline__ void build_a(const float2 (&u)[NCLS][CT][USlots<MT>::QH][4], const StreamArgs& a, int m,
                                        int g, float (&A)[NCLS][CT][MT][4]) {
#pragma unroll
  for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) {
      if constexpr (MT == 1) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          bool is_re;
          const int j = i >> 1;
          const bool ok = u_index<CT, NCLS, TF, MT>(a, m, g, cl, ct, 0, j, &is_re) >= 0;
          const float2 v = ok ? u[cl][ct][0][j] : make_float2(0.f, 0.f);
          A[cl][ct][0][i] = (i & 1) == 0 ? (is_re ? v.x : v.y) : (is_re ? -v.y : v.x);
        }
      } else {
#pragma unroll
        for (int qh = 0; qh < MT / 2; ++qh)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            bool is_re;
            const bool ok = u_index<CT, NCLS, TF, MT>(a, m, g, cl, ct, qh, i, &is_re) >= 0;
            const float2 v = ok ? u[cl][ct][qh][i] : make_float2(0.f, 0.f);
            A[cl][ct][qh][i] = is_re ? v.x : v.y;
            A[cl][ct][qh + MT / 2][i] = is_re ? -v.y : v.x;
          }
      }
    }
}

// t-folded inverse row (CT = 2, N_t = 32 whole) with the three-product
// complex z expansion.  Row r = 4g + i of the z expansion (the MFMA M index)
// is k_t = 2(2g + (i & 1)) + (i >> 1): registers 0, 1 hold even k_t and 2, 3
// odd k_t, which the t fold needs apart.  With U the spectrum and C = Cr + i Ci
// the z basis (K index: 16 modes per block, slot 16qh + 4g + i),
//   k1 = sum (Ur + Ui) Cr,   k2 = sum Ur (Ci - Cr),   k3 = sum Ui (Cr + Ci),
//   Re W = k1 - k3,          Im W = k1 + k2,
// three MFMAs per K step where the four real products took four; Re W and
// Im W sit in the same register of the same lane, so the factors +-i of the
// four-class unfold are swaps of the two arrays.  The t image (A operand of
// the t expansion) holds, at tile ct and register i, part ct (0: Re, 1: -Im)
// of C_t at that k_t.

// k_t of row m (the M index) of the t-folded z expansion.
__device__ __forceinline__ int tfg_kt(int m) { return 2 * (2 * (m >> 2) + (m & 1)) + ((m >> 1) & 1); }

// Spectrum index of (slot 16qh + 4g + i of class cl, k_t of row m), or -1.
template <int NCLS>
__device__ __forceinline__ int tfg_index(const StreamArgs& a, int m, int g, int cl, int qh, int i) {
  const int p = (16 * qh + 4 * g + i) * NCLS + cl;
  const int kt = tfg_kt(m);
  return (p < a.kz && kt < a.kt) ? p * a.kt + kt : -1;
}

template <int MT, int NCLS>
__device__ __forceinline__ void load_u_tfg(const float2* urow, const StreamArgs& a, int m, int g,
                                           float2 (&dst)[NCLS][MT / 2][4]) {
#pragma unroll
  for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
    for (int qh = 0; qh < MT / 2; ++qh)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int idx = tfg_index<NCLS>(a, m, g, cl, qh, i);
        dst[cl][qh][i] = urow[idx < 0 ? 0 : idx];
      }
}
