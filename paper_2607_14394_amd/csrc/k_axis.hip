// Complex contraction along a middle axis (gfx950, fp32 MFMA 16x16x4):
//
//   out[b][k][n] (+)= sum_j basis[k][j] in[b][j][n]
//
// This is one per-dimension partial-DFT step of Sec. V-B: forward y
// (j = y, k = k_y), forward x with the shard-sum accumulate of Eq.
// (dtst_reduce) (j = x, k = k_x), and the inverse expansions over x and y
// with conj(B)^T (Sec. V-A Eq. dtst_inverse, reverse order).  The complex
// product B X, with the basis split into (Re, Im) parts Br, Bi, takes three
// real MFMA products instead of four:
//   k1 = Br (Xr + Xi),   k2 = (Bi - Br) Xr,   k3 = (Br + Bi) Xi,
//   Re = k1 - k3,        Im = k1 + k2,
// with the three basis factors stored in the image (parts 0, 1, 2 of an
// entry) and Xr + Xi formed once per input value; every accumulator is
// lane-local, and so is the epilogue.  The expand kernel (below), which keeps
// its inputs for a whole work item, takes the mirror form k1 = (Br + Bi) Xr,
// k2 = Br (Xi - Xr), k3 = Bi (Xr + Xi) on a two-part image (Re, Im): its
// image is staged per workgroup, where a third part costs more than one
// add per basis value.
//
// Folding (FOLD != 0): when the spatial side of the contraction covers the
// whole even global extent N, exp(-2 pi i k (n + N/2) / N) = (-1)^k
// exp(-2 pi i k n / N).  A forward contraction (FOLD = 1) then feeds the even
// retained modes with in[j] + in[j + N/2] and the odd ones with
// in[j] - in[j + N/2] over j < N/2; an inverse expansion (FOLD = 2) forms the
// even-mode sum E and odd-mode sum O once and writes E + O at n and E - O at
// n + N/2.  Either way the MFMA work halves.  The parity of a retained mode
// equals the parity of its position p, because N is even.
//
// Four-class folding (FOLD 3 forward, FOLD 4 inverse): with N % 4 == 0 and
// an even k_max, k mod 4 equals the position p mod 4 of a retained mode, and
// exp(-2 pi i k (n + q N/4) / N) = (-i)^{k q} exp(-2 pi i k n / N).  Class c
// = p mod 4 then takes a quarter-length contraction over n < N/4: the
// forward feeds class c with S_c[n] = sum_q (-i)^{c q} in[n + q N/4] (from
// the sums and differences of the rows n, n + N/2 and n + N/4, n + 3N/4),
// and the inverse forms the class sums E_c over n < N/4 and writes
// sum_c i^{c q} E_c at n + q N/4.  The MFMA work is a quarter of the direct
// contraction's; used when every class fills whole 16-mode tiles.
//
// Work split: a 256-thread workgroup owns one b, 64*NT consecutive n (16*NT
// per wave) and a block of up to KT 16-row tiles of k.  Every lane streams
// in[b][j][n] for its n with 8-byte loads (16 lanes cover 128 contiguous
// bytes), one 16-row step ahead of the MFMAs that consume it; the basis image
// is read with 16-byte loads that hit in L1/L2, each step's tiles issued
// after the next step's input rows.  The epilogue trades values
// between neighbouring lanes so that every store writes two complex values
// (16 bytes) and each store instruction covers whole 128-byte lines.
#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>

#include "dtst_internal.h"

namespace dtst {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4f mfma(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Hides a value from the optimizer: a load from an address chosen by a
// select would otherwise be split into a branch with one load per arm, and
// the compiler's waits after such a branch cover every outstanding load.
__device__ __forceinline__ void opaque(int64_t& v) { __asm__ volatile("" : "+v"(v)); }

// Value of the neighbouring lane (lane ^ 1) via DPP quad_perm [1, 0, 3, 2].
__device__ __forceinline__ float swap_adjacent(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xf, 0xf, false));
}

struct AxisArgs {
  int64_t nb, total;
  int J, KO, NN, JQ, ktiles, kth, kblocks, nblocks, acc;
  int jh;  // FOLD 1: J/2 (contracted half); FOLD 2: J/2 (modes per class);
           // FOLD 3: J/4 (contracted quarter); FOLD 4: J/4 (modes per class)
  int oh;  // FOLD 2: KO/2 (output half); FOLD 4: KO/4 (output quarter)
};

// Blocks are dispatched round-robin over the 8 XCDs; give each XCD a
// contiguous range of logical tiles so the k blocks that re-read one input
// tile share an L2.
__device__ __forceinline__ int64_t xcd_logical(int64_t bid, int64_t grid) {
  const int64_t per = grid / 8;
  if (bid >= per * 8) return bid;
  return (bid % 8) * per + bid / 8;
}

// Stores the four rows k0 + i (i = 0..3) of one 16-column tile held by this
// lane (row i: value (re[i], im[i]) at column n) with 16-byte stores: even
// lanes write rows 0 and 2, odd lanes rows 1 and 3, each as the pair of
// columns (n & ~1, (n & ~1) + 1).  NN is even, so pairs never straddle the
// end of a row.  rowok(i) says whether row k0 + i exists.  With acc the
// stored values are added to what the output held: pre[h] when the caller
// loaded it earlier (same addresses, h = 0, 1), else read here.
template <class RowPtr, class RowOk>
__device__ __forceinline__ void store_tile(const float (&re)[4], const float (&im)[4], int n, bool nok, int acc,
                                           RowPtr rowptr, RowOk rowok, const float4* pre = nullptr) {
  const bool odd = n & 1;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    // even lanes need their neighbour's rows 2h, odd lanes their neighbour's rows 2h + 1
    const int give = odd ? 2 * h : 2 * h + 1;
    const float rr = swap_adjacent(re[give]);
    const float ri = swap_adjacent(im[give]);
    const int row = odd ? 2 * h + 1 : 2 * h;
    const float4 v = odd ? make_float4(rr, ri, re[row], im[row]) : make_float4(re[row], im[row], rr, ri);
    if (nok && rowok(row)) {
      float4* o = reinterpret_cast<float4*>(rowptr(row) + (n & ~1));
      float4 w = v;
      if (acc) {
        const float4 old = pre ? pre[h] : *o;
        w.x += old.x;
        w.y += old.y;
        w.z += old.z;
        w.w += old.w;
      }
      *o = w;
    }
  }
}

template <int KT, int NT, int FOLD, int ACC>
__global__ void __launch_bounds__(256)
axis_kernel(const float2* __restrict__ in, float2* __restrict__ out, const float4* __restrict__ img,
            AxisArgs a) {
  constexpr int NC = FOLD == 2 ? 2 : 1;                        // input classes loaded per K step
  constexpr int NS = FOLD == 1 ? 2 : (FOLD == 3 ? 4 : 1);      // input rows combined per K index
  static_assert(FOLD != 3 || KT == 4, "four-class tiles: one k tile per class");
  static_assert(FOLD != 4, "four-class inverse runs in axis_expand_kernel");
  const int lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int wave = threadIdx.x >> 6;
  for (int64_t hw = blockIdx.x; hw < a.total; hw += gridDim.x) {
    const int64_t base = (hw / gridDim.x) * gridDim.x;
    const int64_t grid_round = (a.total - base < int64_t(gridDim.x)) ? a.total - base : int64_t(gridDim.x);
    const int64_t L = base + xcd_logical(hw - base, grid_round);
    const int nbk = static_cast<int>(L % a.nblocks);
    const int64_t rest = L / a.nblocks;
    const int kb = static_cast<int>(rest % a.kblocks);
    const int64_t b = rest / a.kblocks;

    const int nw = nbk * (64 * NT) + wave * (16 * NT);  // first column of this wave
    const float2* inb = in + b * int64_t(a.J) * a.NN;
    // Entry read by lanes outside the tile (masked when used): per lane, so
    // that the compiler does not turn the load into a branch with a scalar
    // load of a uniform address for those lanes.
    const int64_t spare = m < int64_t(a.J) * a.NN ? m : 0;

    // K index jj = 16q + 4g + i.  FOLD 0: row jj.  FOLD 1: rows jj and
    // jj + J/2.  FOLD 2: rows 2jj (even modes) and 2jj + 1 (odd modes).
    // FOLD 3: rows jj + s J/4, s = 0..3.
    auto load = [&](int q, float2 (&dst)[NC][NS][NT][4], bool (&ok)[NT][4]) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int jj = 16 * q + 4 * g + i;
          const int n = nw + 16 * nt + m;
          const int lim = FOLD == 0 ? a.J : a.jh;
          const bool v_ok = jj < lim && n < a.NN;
          ok[nt][i] = v_ok;
#pragma unroll
          for (int c = 0; c < NC; ++c)
#pragma unroll
            for (int s = 0; s < NS; ++s) {
              const int row = FOLD == 0 ? jj : (FOLD == 2 ? 2 * jj + c : jj + s * a.jh);
              int64_t idx = v_ok ? int64_t(row) * a.NN + n : spare;
              opaque(idx);
              dst[c][s][nt][i] = inb[idx];
            }
        }
    };

    // FOLD 2 keeps separate even / odd accumulators (index e); k1, k2, k3
    // of the three-product form.
    constexpr int NE = FOLD == 2 ? 2 : 1;
    v4f acc1[NE][KT][NT], acc2[NE][KT][NT], acc3[NE][KT][NT];
#pragma unroll
    for (int e = 0; e < NE; ++e)
#pragma unroll
      for (int kk = 0; kk < KT; ++kk)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          acc1[e][kk][nt] = v4f{0.f, 0.f, 0.f, 0.f};
          acc2[e][kk][nt] = v4f{0.f, 0.f, 0.f, 0.f};
          acc3[e][kk][nt] = v4f{0.f, 0.f, 0.f, 0.f};
        }

    float2 vn[NC][NS][NT][4];
    bool okn[NT][4];
    load(0, vn, okn);

    // Accumulating launches (forward x, the shard sum): fetch the values the
    // output holds now right behind the first input loads, so that read is not
    // a second round trip after the MFMAs.  Output row of tile kt, row i:
    // FOLD 0: 16kt + 4g + i; FOLD 1: mode 2s + c of class c = (kt >= kth),
    // s = 16 (kt - c kth) + 4g + i; FOLD 3: mode 4s + c of class c = kt mod 4,
    // s = 16 (kt / 4) + 4g + i.
    auto out_row = [&](int kt, int i) {
      if (FOLD == 1) {
        const int c = kt >= a.kth ? 1 : 0;
        return 2 * (16 * (kt - c * a.kth) + 4 * g + i) + c;
      }
      if (FOLD == 3) return 4 * (16 * (kt >> 2) + 4 * g + i) + (kt & 3);
      return 16 * kt + 4 * g + i;
    };
    float4 pre[ACC ? KT : 1][ACC ? NT : 1][2];
    if constexpr (ACC) {
      const float2* ob = out + b * int64_t(a.KO) * a.NN;
      // even entry for lanes outside the tile (see spare above)
      const int64_t pspare = (m & 14) + 1 < int64_t(a.KO) * a.NN ? (m & 14) : 0;
#pragma unroll
      for (int kk = 0; kk < KT; ++kk)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int kt = kb * KT + kk;
            const int n = nw + 16 * nt + m;
            const int row = out_row(kt, (n & 1) ? 2 * h + 1 : 2 * h);
            const bool ok = kt < a.ktiles && n < a.NN && row < a.KO;
            int64_t idx = ok ? int64_t(row) * a.NN + (n & ~1) : pspare;
            opaque(idx);
            pre[kk][nt][h] = *reinterpret_cast<const float4*>(ob + idx);
          }
    }
    // Basis tiles of step q (A operands, from L1 / L2): loaded at the end of
    // the previous step, after the input rows of step q + 1 went out, so that
    // waiting for them (the memory counter retires loads in order) never
    // waits for that input prefetch.
    float4 b0[KT][NE], b1[KT][NE], b2[KT][NE];
    auto load_basis = [&](int q) {
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) {
        const int kt = min(kb * KT + kk, a.ktiles - 1);
#pragma unroll
        for (int e = 0; e < NE; ++e) {
          // image: FOLD 2 -> [kt][q][class][part], else [kt][q][part]
          const float4* ip = img + ((int64_t(kt) * a.JQ + q) * NE + e) * 3 * 64 + lane;
          b0[kk][e] = ip[0];
          b1[kk][e] = ip[64];
          b2[kk][e] = ip[128];
        }
      }
    };
    load_basis(0);
    for (int q = 0; q < a.JQ && FOLD == 3; ++q) {
      // class inputs S_c of the four rows n + s J/4 (zero outside the tile):
      // e = x0 + x2, f = x1 + x3, u = x0 - x2, d = x1 - x3;
      // S_0 = e + f, S_2 = e - f, S_1 = u - i d, S_3 = u + i d
      float2 sc[4][NT][4];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float2 x0 = vn[0][0][nt][i], x1 = vn[0][1 % NS][nt][i];
          const float2 x2 = vn[0][2 % NS][nt][i], x3 = vn[0][3 % NS][nt][i];
          const float er = x0.x + x2.x, ei = x0.y + x2.y, fr = x1.x + x3.x, fi = x1.y + x3.y;
          const float ur = x0.x - x2.x, ui = x0.y - x2.y, dr = x1.x - x3.x, di = x1.y - x3.y;
          const bool o = okn[nt][i];
          sc[0][nt][i] = o ? make_float2(er + fr, ei + fi) : make_float2(0.f, 0.f);
          sc[1][nt][i] = o ? make_float2(ur + di, ui - dr) : make_float2(0.f, 0.f);
          sc[2][nt][i] = o ? make_float2(er - fr, ei - fi) : make_float2(0.f, 0.f);
          sc[3][nt][i] = o ? make_float2(ur - di, ui + dr) : make_float2(0.f, 0.f);
        }
      if (q + 1 < a.JQ) load(q + 1, vn, okn);
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) {  // tile kk holds class kk
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            const float2 x = sc[kk & 3][nt][i];
            acc1[0][kk][nt] = mfma(b0[kk][0][i], x.x + x.y, acc1[0][kk][nt]);
            acc2[0][kk][nt] = mfma(b1[kk][0][i], x.x, acc2[0][kk][nt]);
            acc3[0][kk][nt] = mfma(b2[kk][0][i], x.y, acc3[0][kk][nt]);
          }
        }
      }
      if (q + 1 < a.JQ) load_basis(q + 1);
    }
    for (int q = 0; q < a.JQ && FOLD != 3; ++q) {
      // B operands: V[c or fold class][nt][i] as (Xr + Xi, Xr, Xi)
      constexpr int NV = FOLD == 0 ? 1 : 2;
      float vr[NV][NT][4], vi[NV][NT][4], vs[NV][NT][4];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool o = okn[nt][i];
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            float2 x;
            if (FOLD == 1) {
              const float2 p0 = vn[0][0][nt][i], p1 = vn[0][NS - 1][nt][i];
              x = v == 0 ? make_float2(p0.x + p1.x, p0.y + p1.y) : make_float2(p0.x - p1.x, p0.y - p1.y);
            } else {
              x = vn[FOLD == 2 ? v : 0][0][nt][i];
            }
            if (!o) x = make_float2(0.f, 0.f);
            vr[v][nt][i] = x.x;
            vi[v][nt][i] = x.y;
            vs[v][nt][i] = x.x + x.y;
          }
        }
      if (q + 1 < a.JQ) load(q + 1, vn, okn);

#pragma unroll
      for (int kk = 0; kk < KT; ++kk) {
        const int kt = min(kb * KT + kk, a.ktiles - 1);
#pragma unroll
        for (int e = 0; e < NE; ++e) {
          const int v = FOLD == 1 ? (kt >= a.kth ? 1 : 0) : (FOLD == 2 ? e : 0);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
              float xr, xi, xs;
              if (FOLD == 1) {  // uniform select of the fold class of this tile
                xr = v ? vr[NV - 1][nt][i] : vr[0][nt][i];
                xi = v ? vi[NV - 1][nt][i] : vi[0][nt][i];
                xs = v ? vs[NV - 1][nt][i] : vs[0][nt][i];
              } else {
                xr = vr[FOLD == 2 ? e : 0][nt][i];
                xi = vi[FOLD == 2 ? e : 0][nt][i];
                xs = vs[FOLD == 2 ? e : 0][nt][i];
              }
              acc1[e][kk][nt] = mfma(b0[kk][e][i], xs, acc1[e][kk][nt]);
              acc2[e][kk][nt] = mfma(b1[kk][e][i], xr, acc2[e][kk][nt]);
              acc3[e][kk][nt] = mfma(b2[kk][e][i], xi, acc3[e][kk][nt]);
            }
          }
        }
      }
      if (q + 1 < a.JQ) load_basis(q + 1);
    }

#pragma unroll
    for (int kk = 0; kk < KT; ++kk) {
      const int kt = kb * KT + kk;
      if (kt >= a.ktiles) continue;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int n = nw + 16 * nt + m;
        const bool nok = n < a.NN;
        float2* ob = out + b * int64_t(a.KO) * a.NN;
        // Re = k1 - k3, Im = k1 + k2 of accumulator set e
        auto re_of = [&](int e, int i) { return acc1[e][kk][nt][i] - acc3[e][kk][nt][i]; };
        auto im_of = [&](int e, int i) { return acc1[e][kk][nt][i] + acc2[e][kk][nt][i]; };
        if (FOLD == 0) {
          float re[4], im[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            re[i] = re_of(0, i);
            im[i] = im_of(0, i);
          }
          const int k0 = 16 * kt + 4 * g;
          store_tile(re, im, n, nok, ACC, [&](int i) { return ob + int64_t(k0 + i) * a.NN; },
                     [&](int i) { return k0 + i < a.KO; }, ACC ? pre[ACC ? kk : 0][ACC ? nt : 0] : nullptr);
        } else if (FOLD == 3) {
          // tile kt holds class c = kt mod 4, slots s = 16 (kt / 4) + 4g + i, mode p = 4s + c
          float re[4], im[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            re[i] = re_of(0, i);
            im[i] = im_of(0, i);
          }
          const int c = kt & 3;
          const int s0 = 16 * (kt >> 2) + 4 * g;
          store_tile(re, im, n, nok, ACC, [&](int i) { return ob + int64_t(4 * (s0 + i) + c) * a.NN; },
                     [&](int i) { return 4 * (s0 + i) + c < a.KO; }, ACC ? pre[ACC ? kk : 0][ACC ? nt : 0] : nullptr);
        } else if (FOLD == 1) {
          // tile kt holds class c = kt >= kth, slots s = 16 (kt - c kth) + 4g + i, mode p = 2s + c
          float re[4], im[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            re[i] = re_of(0, i);
            im[i] = im_of(0, i);
          }
          const int c = kt >= a.kth ? 1 : 0;
          const int s0 = 16 * (kt - c * a.kth) + 4 * g;
          store_tile(re, im, n, nok, ACC, [&](int i) { return ob + int64_t(2 * (s0 + i) + c) * a.NN; },
                     [&](int i) { return 2 * (s0 + i) + c < a.KO; }, ACC ? pre[ACC ? kk : 0][ACC ? nt : 0] : nullptr);
        } else {
          // rows y = 16kt + 4g + i < KO/2: E + O at y, E - O at y + KO/2
          const int y0 = 16 * kt + 4 * g;
#pragma unroll
          for (int hf = 0; hf < 2; ++hf) {
            float re[4], im[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float er = re_of(0, i), ei = im_of(0, i);
              const float odr = re_of(NE - 1, i), odi = im_of(NE - 1, i);
              re[i] = hf == 0 ? er + odr : er - odr;
              im[i] = hf == 0 ? ei + odi : ei - odi;
            }
            store_tile(re, im, n, nok, ACC,
                       [&](int i) { return ob + int64_t(y0 + i + hf * a.oh) * a.NN; },
                       [&](int i) { return y0 + i < a.oh; });
          }
        }
      }
    }
  }
}

// Persistent, software-pipelined form of the forward-direction contraction
// (FOLD 0, 1 or 3, no accumulate) for launches whose basis image fits in
// LDS.  A grid of resident workgroups walks its work items (b, k block,
// column block) in order; every wave runs one flat sequence of (item, K
// step) positions and keeps the input rows of the next PD positions in
// flight, across item boundaries, so the first steps of an item are loaded
// while the previous item is still being contracted and written (a work
// item of a short contraction, J = 64 for instance, is only four K steps:
// one workgroup per item would expose the input latency at every item
// start).  The image is copied to LDS once per workgroup; its reads then
// never wait behind input loads or output stores (global loads and stores
// share one memory counter per wave, LDS reads do not).  Buffer k holds
// positions k, k + PD, ...; the loop runs whole passes over the buffers so
// every buffer index is a compile-time constant.  Loads past the last
// position re-read the last item's rows and are never used.
template <int KT, int NT, int FOLD>
__global__ void __launch_bounds__(256)
axis_pipe_kernel(const float2* __restrict__ in, float2* __restrict__ out, const float4* __restrict__ img,
                 AxisArgs a) {
  static_assert(FOLD == 0 || FOLD == 1 || FOLD == 3, "forward-direction folds only");
  static_assert(FOLD != 3 || KT == 4, "four-class tiles: one k tile per class");
  constexpr int NS = FOLD == 1 ? 2 : (FOLD == 3 ? 4 : 1);  // input rows combined per K index
  constexpr int PD = 2;
  extern __shared__ float4 simg[];
  const int lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int wave = threadIdx.x >> 6;
  const int64_t G = gridDim.x;
  const int64_t n_it = a.total > int64_t(blockIdx.x) ? (a.total - 1 - blockIdx.x) / G + 1 : 0;
  if (n_it == 0) return;
  const int lim = FOLD == 0 ? a.J : a.jh;
  const int64_t spare = m < int64_t(a.J) * a.NN ? m : 0;

  // work item `it` of this workgroup -> (b, k block, first column of this
  // wave); items of one round of the grid are spread over the XCDs in
  // contiguous logical ranges (as in axis_kernel)
  struct Item {
    int64_t b;
    int kb, nw;
  };
  // (32-bit index arithmetic: the launcher takes this kernel only for fewer
  // than 2^31 work items)
  auto item_of = [&](int64_t it) {
    const uint32_t g32 = static_cast<uint32_t>(G), tot = static_cast<uint32_t>(a.total);
    const uint32_t base = static_cast<uint32_t>(it) * g32;
    const uint32_t grid_round = tot - base < g32 ? tot - base : g32;
    const uint32_t per = grid_round / 8, bid = blockIdx.x;
    const uint32_t L = base + (bid >= per * 8 ? bid : (bid % 8) * per + bid / 8);
    const uint32_t nbl = static_cast<uint32_t>(a.nblocks), kbl = static_cast<uint32_t>(a.kblocks);
    Item r;
    const uint32_t rest = L / nbl;
    const int nbk = static_cast<int>(L - rest * nbl);
    const uint32_t b = rest / kbl;
    r.kb = static_cast<int>(rest - b * kbl);
    r.b = b;
    r.nw = nbk * (64 * NT) + wave * (16 * NT);
    return r;
  };

  float2 vb[PD][NS][NT][4];
  bool okb[PD][NT][4];
  // load position (item, step) and its item
  int64_t it_l = 0;
  int q_l = 0;
  Item t_l = item_of(0);
  auto load = [&](auto kc) __attribute__((always_inline)) {
    constexpr int k = decltype(kc)::value;
    const float2* inb = in + t_l.b * int64_t(a.J) * a.NN;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int jj = 16 * q_l + 4 * g + i;
        const int n = t_l.nw + 16 * nt + m;
        const bool v_ok = jj < lim && n < a.NN;
        okb[k][nt][i] = v_ok;
#pragma unroll
        for (int sr = 0; sr < NS; ++sr) {
          int64_t idx = v_ok ? int64_t(jj + sr * (FOLD == 0 ? 0 : a.jh)) * a.NN + n : spare;
          opaque(idx);
          vb[k][sr][nt][i] = inb[idx];
        }
      }
    if (++q_l == a.JQ) {
      q_l = 0;
      if (it_l + 1 < n_it) t_l = item_of(++it_l);
    }
  };
  load(std::integral_constant<int, 0>{});
  load(std::integral_constant<int, 1>{});
  {
    const int n4 = a.ktiles * a.JQ * 3 * 64;
    for (int e = threadIdx.x; e < n4; e += 256) simg[e] = img[e];
  }
  __syncthreads();

  v4f acc1[KT][NT], acc2[KT][NT], acc3[KT][NT];
  auto clear = [&]() {
#pragma unroll
    for (int kk = 0; kk < KT; ++kk)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        acc1[kk][nt] = v4f{0.f, 0.f, 0.f, 0.f};
        acc2[kk][nt] = v4f{0.f, 0.f, 0.f, 0.f};
        acc3[kk][nt] = v4f{0.f, 0.f, 0.f, 0.f};
      }
  };
  clear();

  // compute position
  int64_t it_c = 0;
  int q_c = 0;
  Item t_c = item_of(0);

  auto step = [&](auto kc) __attribute__((always_inline)) {
    constexpr int k = decltype(kc)::value;
    const bool live = it_c < n_it;
    // class inputs of this position: V[v][nt][i] (v = fold class of a tile;
    // FOLD 3: S_c as in axis_kernel, zero outside the tile)
    constexpr int NV = FOLD == 0 ? 1 : (FOLD == 1 ? 2 : 4);
    float2 xv[NV][NT][4];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool o = okb[k][nt][i];
        const float2 x0 = vb[k][0][nt][i];
        if (FOLD == 0) {
          xv[0][nt][i] = o ? x0 : make_float2(0.f, 0.f);
        } else if (FOLD == 1) {
          const float2 x1 = vb[k][NS - 1][nt][i];
          xv[0][nt][i] = o ? make_float2(x0.x + x1.x, x0.y + x1.y) : make_float2(0.f, 0.f);
          xv[NV - 1][nt][i] = o ? make_float2(x0.x - x1.x, x0.y - x1.y) : make_float2(0.f, 0.f);
        } else {
          const float2 x1 = vb[k][1 % NS][nt][i], x2 = vb[k][2 % NS][nt][i], x3 = vb[k][3 % NS][nt][i];
          const float er = x0.x + x2.x, ei = x0.y + x2.y, fr = x1.x + x3.x, fi = x1.y + x3.y;
          const float ur = x0.x - x2.x, ui = x0.y - x2.y, dr = x1.x - x3.x, di = x1.y - x3.y;
          xv[0][nt][i] = o ? make_float2(er + fr, ei + fi) : make_float2(0.f, 0.f);
          xv[1 % NV][nt][i] = o ? make_float2(ur + di, ui - dr) : make_float2(0.f, 0.f);
          xv[2 % NV][nt][i] = o ? make_float2(er - fr, ei - fi) : make_float2(0.f, 0.f);
          xv[3 % NV][nt][i] = o ? make_float2(ur - di, ui + dr) : make_float2(0.f, 0.f);
        }
      }
    load(kc);
    if (!live) return;
    float4 b0[KT], b1[KT], b2[KT];
#pragma unroll
    for (int kk = 0; kk < KT; ++kk) {
      const int kt = min(t_c.kb * KT + kk, a.ktiles - 1);
      const int ie = (kt * a.JQ + q_c) * 3 * 64 + lane;
      b0[kk] = simg[ie];
      b1[kk] = simg[ie + 64];
      b2[kk] = simg[ie + 128];
    }
    // i outermost: consecutive products into one accumulator are 3 KT NT
    // instructions apart
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) {
        const int kt = min(t_c.kb * KT + kk, a.ktiles - 1);
        // fold class of tile kt: FOLD 1 (kt >= kth), FOLD 3 (kt mod 4 = kk)
        const int v = FOLD == 1 ? (kt >= a.kth ? 1 : 0) : (FOLD == 3 ? (kk & 3) : 0);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          float2 x;
          if (FOLD == 1) x = v ? xv[NV - 1][nt][i] : xv[0][nt][i];  // uniform select
          else x = xv[FOLD == 3 ? (kk & 3) % NV : 0][nt][i];
          acc1[kk][nt] = mfma(b0[kk][i], x.x + x.y, acc1[kk][nt]);
          acc2[kk][nt] = mfma(b1[kk][i], x.x, acc2[kk][nt]);
          acc3[kk][nt] = mfma(b2[kk][i], x.y, acc3[kk][nt]);
        }
      }
    if (++q_c < a.JQ) return;
    // item finished: Re = k1 - k3, Im = k1 + k2 of every tile, rows as in axis_kernel
    float2* ob = out + t_c.b * int64_t(a.KO) * a.NN;
#pragma unroll
    for (int kk = 0; kk < KT; ++kk) {
      const int kt = t_c.kb * KT + kk;
      if (kt >= a.ktiles) continue;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int n = t_c.nw + 16 * nt + m;
        float re[4], im[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          re[i] = acc1[kk][nt][i] - acc3[kk][nt][i];
          im[i] = acc1[kk][nt][i] + acc2[kk][nt][i];
        }
        auto row = [&](int i) {
          if (FOLD == 1) {
            const int c = kt >= a.kth ? 1 : 0;
            return 2 * (16 * (kt - c * a.kth) + 4 * g + i) + c;
          }
          if (FOLD == 3) return 4 * (16 * (kt >> 2) + 4 * g + i) + (kt & 3);
          return 16 * kt + 4 * g + i;
        };
        store_tile(re, im, n, n < a.NN, 0, [&](int i) { return ob + int64_t(row(i)) * a.NN; },
                   [&](int i) { return row(i) < a.KO; });
      }
    }
    clear();
    q_c = 0;
    if (++it_c < n_it) t_c = item_of(it_c);
  };
  static_assert(PD == 2, "two positions in flight");
  do {
    step(std::integral_constant<int, 0>{});
    step(std::integral_constant<int, 1>{});
  } while (it_c < n_it);
}

// Folded inverse expansion (FOLD 2 with NCL = 2 classes, FOLD 4 with NCL =
// 4) whose whole contraction fits in a few K steps (JQ <= 2: at most 32
// retained modes per class).  Such a launch writes several times what it
// reads (N rows from K modes), so each workgroup loads its input columns
// once, keeps them in registers and loops over every block of KT output
// tiles: the stores of one block overlap the products of the next, and no
// other workgroup re-reads the input.  KT output tiles per block (one 16-row
// tile of the N/NCL rows of a class sum), NT 16-column tiles per wave.
// LI: the basis image is copied to LDS once per workgroup, right behind the
// first input loads.  Global loads and stores share a wave's memory counter,
// so image reads from global memory inside the loop would wait for the
// previous block's stores to complete; LDS reads do not.
template <int KT, int NT, int JQ, int NCL, int LI>
__global__ void __launch_bounds__(256)
axis_expand_kernel(const float2* __restrict__ in, float2* __restrict__ out, const float4* __restrict__ img,
                   AxisArgs a) {
  extern __shared__ float4 simg[];
  const int lane = threadIdx.x & 63;
  const int m = lane & 15, g = lane >> 4;
  const int wave = threadIdx.x >> 6;
  const int64_t total = a.total;
  bool staged = false;
  for (int64_t hw = blockIdx.x; hw < total; hw += gridDim.x) {
    const int64_t base = (hw / gridDim.x) * gridDim.x;
    const int64_t grid_round = (total - base < int64_t(gridDim.x)) ? total - base : int64_t(gridDim.x);
    const int64_t L = base + xcd_logical(hw - base, grid_round);
    const int nbk = static_cast<int>(L % a.nblocks);
    const int64_t b = L / a.nblocks;
    const int nw = nbk * (64 * NT) + wave * (16 * NT);
    const float2* inb = in + b * int64_t(a.J) * a.NN;
    float2* ob = out + b * int64_t(a.KO) * a.NN;
    const int64_t spare = m < int64_t(a.J) * a.NN ? m : 0;

    // K index jj = 16q + 4g + i: row NCL jj + c (mode of class c); the B
    // operands of the three products, Xr, Xi - Xr and Xr + Xi, are formed
    // once per work item (every output tile reuses them)
    float2 x[JQ][NCL][NT][4];
#pragma unroll
    for (int q = 0; q < JQ; ++q)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int jj = 16 * q + 4 * g + i;
          const int n = nw + 16 * nt + m;
          const bool ok = jj < a.jh && n < a.NN;
#pragma unroll
          for (int c = 0; c < NCL; ++c) {
            int64_t idx = ok ? int64_t(NCL * jj + c) * a.NN + n : spare;
            opaque(idx);
            const float2 v = inb[idx];
            x[q][c][nt][i] = ok ? v : make_float2(0.f, 0.f);
          }
        }
    if (LI && !staged) {
      const int n4 = a.ktiles * JQ * NCL * 2 * 64;
      for (int e = threadIdx.x; e < n4; e += 256) simg[e] = img[e];
      __syncthreads();
      staged = true;
    }
    float xr[JQ][NCL][NT][4], xd[JQ][NCL][NT][4], xs[JQ][NCL][NT][4];
#pragma unroll
    for (int q = 0; q < JQ; ++q)
#pragma unroll
      for (int c = 0; c < NCL; ++c)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float2 v = x[q][c][nt][i];
            xr[q][c][nt][i] = v.x;
            xd[q][c][nt][i] = v.y - v.x;
            xs[q][c][nt][i] = v.x + v.y;
          }

    for (int kb = 0; kb < a.kblocks; ++kb) {
      v4f acc1[NCL][KT][NT], acc2[NCL][KT][NT], acc3[NCL][KT][NT];
#pragma unroll
      for (int e = 0; e < NCL; ++e)
#pragma unroll
        for (int kk = 0; kk < KT; ++kk)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            acc1[e][kk][nt] = v4f{0.f, 0.f, 0.f, 0.f};
            acc2[e][kk][nt] = v4f{0.f, 0.f, 0.f, 0.f};
            acc3[e][kk][nt] = v4f{0.f, 0.f, 0.f, 0.f};
          }
#pragma unroll
      for (int q = 0; q < JQ; ++q) {
        float4 bre[KT][NCL], bim[KT][NCL];
#pragma unroll
        for (int kk = 0; kk < KT; ++kk) {
          const int kt = min(kb * KT + kk, a.ktiles - 1);
#pragma unroll
          for (int e = 0; e < NCL; ++e) {
            // image entry (((kt * JQ + q) * NCL + class) * 2 + part) * 64 + lane
            const int ie = ((kt * JQ + q) * NCL + e) * 2 * 64 + lane;
            bre[kk][e] = LI ? simg[ie] : img[ie];
            bim[kk][e] = LI ? simg[ie + 64] : img[ie + 64];
          }
        }
#pragma unroll
        for (int kk = 0; kk < KT; ++kk)
#pragma unroll
          for (int e = 0; e < NCL; ++e)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float r = bre[kk][e][i], im = bim[kk][e][i], rpi = r + im;
#pragma unroll
              for (int nt = 0; nt < NT; ++nt) {
                acc1[e][kk][nt] = mfma(rpi, xr[q][e][nt][i], acc1[e][kk][nt]);
                acc2[e][kk][nt] = mfma(r, xd[q][e][nt][i], acc2[e][kk][nt]);
                acc3[e][kk][nt] = mfma(im, xs[q][e][nt][i], acc3[e][kk][nt]);
              }
            }
      }
      // rows y = 16kt + 4g + i < KO/NCL of the class sums E_c (Re = k1 - k3,
      // Im = k1 + k2).  NCL 2: E_0 + E_1 at y, E_0 - E_1 at y + KO/2.  NCL 4:
      // with P = E_0 + E_2, Q = E_0 - E_2, R = E_1 + E_3, T = E_1 - E_3, the
      // rows y + h KO/4 get P + R, Q + i T, P - R, Q - i T (h = 0..3).
#pragma unroll
      for (int kk = 0; kk < KT; ++kk) {
        const int kt = kb * KT + kk;
        if (kt >= a.ktiles) continue;
        const int y0 = 16 * kt + 4 * g;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int n = nw + 16 * nt + m;
          const bool nok = n < a.NN;
          auto er = [&](int e, int i) { return acc1[e][kk][nt][i] - acc3[e][kk][nt][i]; };
          auto ei = [&](int e, int i) { return acc1[e][kk][nt][i] + acc2[e][kk][nt][i]; };
#pragma unroll
          for (int hf = 0; hf < NCL; ++hf) {
            float re[4], im[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              if (NCL == 2) {
                re[i] = hf == 0 ? er(0, i) + er(NCL - 1, i) : er(0, i) - er(NCL - 1, i);
                im[i] = hf == 0 ? ei(0, i) + ei(NCL - 1, i) : ei(0, i) - ei(NCL - 1, i);
              } else {
                const int c2 = 2 % NCL, c3 = 3 % NCL;
                if (hf == 0 || hf == 2) {
                  const float pr = er(0, i) + er(c2, i), pi = ei(0, i) + ei(c2, i);
                  const float rr = er(1, i) + er(c3, i), ri = ei(1, i) + ei(c3, i);
                  re[i] = hf == 0 ? pr + rr : pr - rr;
                  im[i] = hf == 0 ? pi + ri : pi - ri;
                } else {
                  const float qr = er(0, i) - er(c2, i), qi = ei(0, i) - ei(c2, i);
                  const float tr = er(1, i) - er(c3, i), ti = ei(1, i) - ei(c3, i);
                  re[i] = hf == 1 ? qr - ti : qr + ti;
                  im[i] = hf == 1 ? qi + tr : qi - tr;
                }
              }
            }
            store_tile(re, im, n, nok, 0, [&](int i) { return ob + int64_t(y0 + i + hf * a.oh) * a.NN; },
                       [&](int i) { return y0 + i < a.oh; });
          }
        }
      }
    }
  }
}

// LDS bytes of an expand kernel's staged basis image (ncl classes per
// entry, two parts), or 0 when the image is larger than 32 KiB and is read
// from global memory instead (two workgroups of the expand kernels share a
// CU, and each one stages the image for its single work item).
size_t expand_lds_bytes(const AxisCfg& c, int ncl) {
  const size_t b = size_t(c.ktiles) * c.JQ * ncl * 2 * 64 * sizeof(float4);
  return b <= 32 * 1024 ? b : 0;
}

typedef void (*axis_fn)(const float2*, const float2*, float2*, const float4*, AxisArgs);

// Workgroups of kernel f with `lds` bytes of dynamic LDS the current device
// holds at once (cached per kernel, LDS size and device).
int64_t resident(const void* f, size_t lds) {
  struct Entry {
    const void* f;
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

// The persistent pipelined kernel for (KT, NT, FOLD).
template <int FOLD>
const void* pipe_fn(int kt, int nt) {
  if (FOLD == 3) return reinterpret_cast<const void*>(axis_pipe_kernel<4, 1, 3>);
  if (kt == 1) return nt == 2 ? reinterpret_cast<const void*>(axis_pipe_kernel<1, 2, FOLD == 3 ? 0 : FOLD>)
                              : reinterpret_cast<const void*>(axis_pipe_kernel<1, 1, FOLD == 3 ? 0 : FOLD>);
  if (kt == 2) return nt == 2 ? reinterpret_cast<const void*>(axis_pipe_kernel<2, 2, FOLD == 3 ? 0 : FOLD>)
                              : reinterpret_cast<const void*>(axis_pipe_kernel<2, 1, FOLD == 3 ? 0 : FOLD>);
  return nt == 2 ? reinterpret_cast<const void*>(axis_pipe_kernel<4, 2, FOLD == 3 ? 0 : FOLD>)
                 : reinterpret_cast<const void*>(axis_pipe_kernel<4, 1, FOLD == 3 ? 0 : FOLD>);
}

// Launches the pipelined kernel when its image fits 64 KiB of LDS; returns
// false (nothing launched) otherwise.
bool launch_pipe(int fold, int kt, int nt, const AxisCfg& c, AxisArgs a, hipStream_t s, const float2* pin,
                 float2* pout, const float4* pimg, hipError_t* err) {
  const size_t lds = size_t(c.ktiles) * c.JQ * 3 * 64 * sizeof(float4);
  if (lds > 64 * 1024 || a.nb * a.kblocks * ((c.NN + 63) / 64) >= (int64_t(1) << 31)) return false;
  // four k tiles keep twelve accumulator tiles per column tile: one column
  // tile per wave (two would leave one wave per SIMD)
  if (kt == 4) nt = 1;
  if (nt == 1) {
    a.nblocks = (c.NN + 63) / 64;
    a.total = a.nb * a.kblocks * a.nblocks;
  }
  const void* f = fold == 0 ? pipe_fn<0>(kt, nt) : (fold == 1 ? pipe_fn<1>(kt, nt) : pipe_fn<3>(kt, nt));
  const int64_t res = resident(f, lds);
  if (res <= 0) {
    *err = hipErrorInvalidConfiguration;
    return true;
  }
  const int grid = static_cast<int>(a.total < res ? a.total : res);
  void* args[] = {&pin, &pout, &pimg, &a};
  *err = hipLaunchKernel(f, dim3(grid), dim3(256), args, lds, s);
  return true;
}

template <int KT, int FOLD, int ACC>
void launch_kt(int nt, int grid, hipStream_t s, const float2* pin, float2* pout, const float4* pimg,
               const AxisArgs& a) {
  if (nt == 2)
    hipLaunchKernelGGL((axis_kernel<KT, 2, FOLD, ACC>), dim3(grid), dim3(256), 0, s, pin, pout, pimg, a);
  else
    hipLaunchKernelGGL((axis_kernel<KT, 1, FOLD, ACC>), dim3(grid), dim3(256), 0, s, pin, pout, pimg, a);
}

template <int FOLD, int ACC>
void launch_fold(int kt, int nt, int grid, hipStream_t s, const float2* pin, float2* pout, const float4* pimg,
                 const AxisArgs& a) {
  if (kt == 1) launch_kt<1, FOLD, ACC>(nt, grid, s, pin, pout, pimg, a);
  else if (kt == 2) launch_kt<2, FOLD, ACC>(nt, grid, s, pin, pout, pimg, a);
  else launch_kt<4, FOLD, ACC>(nt, grid, s, pin, pout, pimg, a);
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
  a.kth = c.kth;
  const int ncls = (c.fold == 3 || c.fold == 4) ? 4 : 2;
  a.jh = c.J / ncls;
  a.oh = c.KO / ncls;
  a.acc = accumulate ? 1 : 0;
  // FOLD 2 keeps two accumulator sets; cap its k block at 2 tiles.
  const int kmax = c.fold == 2 ? 2 : 4;
  int kt = c.ktiles <= 1 ? 1 : (c.ktiles <= 2 || kmax == 2 ? 2 : 4);
  a.kblocks = (c.ktiles + kt - 1) / kt;
  // Two 16-column tiles per wave when that still leaves several workgroups per CU.
  int nt = 2;
  if (nb * a.kblocks * ((c.NN + 127) / 128) < 2048) nt = 1;
  a.nblocks = (c.NN + 64 * nt - 1) / (64 * nt);
  a.total = nb * a.kblocks * a.nblocks;
  const int64_t cap = int64_t(1) << 22;
  const int grid = static_cast<int>(a.total < cap ? a.total : cap);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const float2* pin = static_cast<const float2*>(in);
  float2* pout = static_cast<float2*>(out);
  const float4* pimg = reinterpret_cast<const float4*>(img);
  // Accumulation only happens on forward-direction launches (fold 0, 1, 3).
  if ((c.fold == 2 || c.fold == 4) && a.acc) return hipErrorInvalidValue;
  // image parts the kernel taking this launch reads: (Re, Im) for the expand
  // kernel, (Br, Bi - Br, Br + Bi) for the others
  const bool expand = (c.fold == 2 || c.fold == 4) && c.JQ <= 2;
  if (c.parts != (expand ? 2 : 3)) return hipErrorInvalidValue;
  if (c.fold == 3) {
    // one k tile per class in every block (KT = 4), one 16-column tile per
    // wave (the four class inputs and twelve accumulator tiles of NT = 2
    // would not fit the registers of two waves per SIMD)
    if (c.ktiles % 4 != 0) return hipErrorInvalidValue;
    AxisArgs f = a;
    f.kblocks = c.ktiles / 4;
    f.nblocks = (c.NN + 63) / 64;
    f.total = nb * f.kblocks * f.nblocks;
    const int g3 = static_cast<int>(f.total < cap ? f.total : cap);
    hipError_t perr = hipSuccess;
    if (!f.acc && launch_pipe(3, 4, 1, c, f, s, pin, pout, pimg, &perr)) return perr;
    if (f.acc) hipLaunchKernelGGL((axis_kernel<4, 1, 3, 1>), dim3(g3), dim3(256), 0, s, pin, pout, pimg, f);
    else hipLaunchKernelGGL((axis_kernel<4, 1, 3, 0>), dim3(g3), dim3(256), 0, s, pin, pout, pimg, f);
    return hipGetLastError();
  }
  if (c.fold == 4) {
    // the four class sums of one output tile per block, the contraction in
    // one or two K steps (at most 32 modes per class), one 16-column tile per
    // wave (two would hold twice the inputs and accumulators: one wave per
    // SIMD)
    if (c.JQ > 2) return hipErrorInvalidValue;
    AxisArgs e = a;
    e.kblocks = c.ktiles;
    e.nblocks = (c.NN + 63) / 64;
    e.total = nb * e.nblocks;
    const int g4 = static_cast<int>(e.total < cap ? e.total : cap);
    const size_t lds = expand_lds_bytes(c, 4);
    if (lds > 0) {
      if (c.JQ == 1) hipLaunchKernelGGL((axis_expand_kernel<1, 1, 1, 4, 1>), dim3(g4), dim3(256), lds, s, pin, pout, pimg, e);
      else hipLaunchKernelGGL((axis_expand_kernel<1, 1, 2, 4, 1>), dim3(g4), dim3(256), lds, s, pin, pout, pimg, e);
    } else {
      if (c.JQ == 1) hipLaunchKernelGGL((axis_expand_kernel<1, 1, 1, 4, 0>), dim3(g4), dim3(256), 0, s, pin, pout, pimg, e);
      else hipLaunchKernelGGL((axis_expand_kernel<1, 1, 2, 4, 0>), dim3(g4), dim3(256), 0, s, pin, pout, pimg, e);
    }
    return hipGetLastError();
  }
  if (c.fold == 2 && c.JQ <= 2) {
    // The whole contraction in registers; every workgroup loops over all k
    // tiles one at a time (measured fastest at the backward workload's
    // 64-mode y expansion against blocks of two or four tiles), so the work
    // items are (b, column block) only.
    AxisArgs e = a;
    e.kblocks = c.ktiles;
    const int ent = nb * ((c.NN + 127) / 128) < 2048 ? 1 : 2;
    e.nblocks = (c.NN + 64 * ent - 1) / (64 * ent);
    e.total = nb * e.nblocks;
    const int g2 = static_cast<int>(e.total < cap ? e.total : cap);
    const size_t lds = expand_lds_bytes(c, 2);
    if (lds > 0) {
      if (c.JQ == 1) {
        if (ent == 2) hipLaunchKernelGGL((axis_expand_kernel<1, 2, 1, 2, 1>), dim3(g2), dim3(256), lds, s, pin, pout, pimg, e);
        else hipLaunchKernelGGL((axis_expand_kernel<1, 1, 1, 2, 1>), dim3(g2), dim3(256), lds, s, pin, pout, pimg, e);
      } else {
        if (ent == 2) hipLaunchKernelGGL((axis_expand_kernel<1, 2, 2, 2, 1>), dim3(g2), dim3(256), lds, s, pin, pout, pimg, e);
        else hipLaunchKernelGGL((axis_expand_kernel<1, 1, 2, 2, 1>), dim3(g2), dim3(256), lds, s, pin, pout, pimg, e);
      }
    } else if (c.JQ == 1) {
      if (ent == 2) hipLaunchKernelGGL((axis_expand_kernel<1, 2, 1, 2, 0>), dim3(g2), dim3(256), 0, s, pin, pout, pimg, e);
      else hipLaunchKernelGGL((axis_expand_kernel<1, 1, 1, 2, 0>), dim3(g2), dim3(256), 0, s, pin, pout, pimg, e);
    } else {
      if (ent == 2) hipLaunchKernelGGL((axis_expand_kernel<1, 2, 2, 2, 0>), dim3(g2), dim3(256), 0, s, pin, pout, pimg, e);
      else hipLaunchKernelGGL((axis_expand_kernel<1, 1, 2, 2, 0>), dim3(g2), dim3(256), 0, s, pin, pout, pimg, e);
    }
    return hipGetLastError();
  }
  if (c.fold != 2 && !a.acc) {
    hipError_t perr = hipSuccess;
    if (launch_pipe(c.fold, kt, nt, c, a, s, pin, pout, pimg, &perr)) return perr;
  }
  if (c.fold == 2) launch_fold<2, 0>(kt, nt, grid, s, pin, pout, pimg, a);
  else if (c.fold == 1) a.acc ? launch_fold<1, 1>(kt, nt, grid, s, pin, pout, pimg, a)
                              : launch_fold<1, 0>(kt, nt, grid, s, pin, pout, pimg, a);
  else a.acc ? launch_fold<0, 1>(kt, nt, grid, s, pin, pout, pimg, a)
             : launch_fold<0, 0>(kt, nt, grid, s, pin, pout, pimg, a);
  return hipGetLastError();
}

}  // namespace dtst
