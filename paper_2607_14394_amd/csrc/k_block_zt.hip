// Inverse z + t expansion fused with the block epilogue (Sec. V "Block
// Structure"; Algorithm 1, its first and last step):
//
//   y[b,o,n] = GELU( sum_i w[o,i] x[b,i,n] + Re sum_{kz,kt} C_t C_z V[b,o,kz,kt] ),
//
// where V is the y-expanded spectrum (B, C_out, N_x, N_y, K_z, K_t) of the
// inverse chain and C_z, C_t the z and t expansion bases (half-spectrum
// weights and 1/prod N folded into C_t).  The separate epilogue kernel reads
// y back and writes it again; here every output value is written once and
// the layer input x is read once.
//
// A workgroup of kBlkWaves waves owns one (b, x, y) row at a time
// (persistent over rows) and produces every output channel of it, one chunk
// at a time: a chunk is the 16 z rows of one z tile of one fold class (all
// N_t of them), so a z tile of a folded row is two chunks.
//   phase 1: wave w expands the chunk for the channels o = w, w + kBlkWaves,
//            ... from the row's spectrum (staged in LDS for every channel at
//            the row start): the z expansion and class unfold once per z
//            tile (kept in registers for the tile's second chunk), the t
//            expansion of the chunk's class; the values go to one of two LDS
//            buffers as [o][z row][t];
//   phase 2: wave w takes one 64-point group of the chunk and forms
//            y[o][p] = GELU(Ys[o][p] + sum_i w[o,i] x[i][p]) on the matrix
//            cores: M = output channel (16 per tile), N = point, K = input
//            channel, the accumulators starting from the expanded values read
//            back from LDS.  Lane (g, m) holds points 4m..4m+3 of the group
//            (N tile j = point 4m + j), so the x loads and the output stores
//            are 16-byte accesses of 16 consecutive lanes over 256 bytes of
//            one channel.  x is loaded NCLS chunks ahead.
// With two buffers, phase 1 of the next chunk writes the buffer phase 2 of
// the previous chunk has finished reading: one barrier per chunk.
// MFMA 16x16x4 fp32 lane layout (lane l, m = l & 15, g = l >> 4):
//   A operand A[m][g], B operand B[g][m], accumulator register i: C[4g+i][m].
#include <hip/hip_runtime.h>

#include <type_traits>

#include "dtst_internal.h"

namespace dtst {
namespace {

#include "stream_ops.h"

// A chunk has 16 z rows of at most 32 t: at most 8 groups of 64 points, one
// per wave.
constexpr int kBlkWaves = 8;

#include "gelu_as.h"

struct BlockArgs {
  int64_t rows;  // B * N_x * N_y
  int64_t xy;    // N_x * N_y
  int ci, co;
  int groups;    // 64-point groups per chunk: N_t / 4
  int ostride;   // LDS floats per output channel of a buffer: 16 * N_t
};

// Float offset of (z row zr, t) in a channel of an LDS value buffer.  With
// N_t = 32 the 16-byte t chunk index is XORed with bits 1..3 of the z row, so
// that the 16 z rows one MFMA tile writes (one row per lane) spread over the
// banks instead of two rows of 128 bytes sharing them.
__device__ __forceinline__ int yoff(int zr, int t, int nt) {
  return nt == 32 ? zr * 32 + (t ^ (((zr >> 1) & 7) << 2)) : zr * nt + t;
}

// z expansion and class unfold of one z tile for one channel's row (the
// t-expansion operands of the tile's chunks), unfolded t.
template <int CT, int MT, int NCLS>
__device__ __forceinline__ void zexp_plain(const float2* urow, const StreamArgs& a, const float4 (&Bz)[NCLS][MT],
                                           int m, int g, v4f (&W)[NCLS][CT]) {
  float2 un[NCLS][CT][USlots<MT>::QH][4];
  load_u<CT, MT, NCLS>(urow, a, m, g, un);
  float A[NCLS][CT][MT][4];
  build_a<CT, MT, NCLS>(un, a, m, g, A);
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
        for (int ct = 0; ct < CT; ++ct) W[cl][ct] = mfma(A[cl][ct][q][i], Bz[cl][q][i], W[cl][ct]);
  unfold_classes<NCLS, CT>(W);
}

// t expansion of one class of a z tile (unfolded t) into yb[z row][t].
template <int CT, int TH, bool WHOLE_T = false>
__device__ __forceinline__ void texp_plain(const v4f (&W)[CT], const float (&ta)[TH][CT][4], float* yb, int nt,
                                           int m, int g) {
  v4f Y[TH];
#pragma unroll
  for (int mt = 0; mt < TH; ++mt) Y[mt] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int mt = 0; mt < TH; ++mt) Y[mt] = mfma(ta[mt][ct][i], W[ct][i], Y[mt]);
#pragma unroll
  for (int mt = 0; mt < TH; ++mt) {
    const int t0 = 16 * mt + 4 * g;
    if (WHOLE_T || t0 < nt) *reinterpret_cast<v4f*>(yb + yoff(m, t0, nt)) = Y[mt];
  }
}

// t folded (CT = 2, N_t = 32 whole): the three-product z expansion of
// inv_row_tfg for one z tile and the class unfold; Re and Im of the
// expanded values in separate arrays.
template <int MT, int NCLS>
__device__ __forceinline__ void zexp_tfg(const float2* urow, const StreamArgs& a, const float4* lz, int zt, int m,
                                         int g, int lane, v4f (&Wr)[NCLS], v4f (&Wi)[NCLS]) {
  float2 u[NCLS][MT / 2][4];
  load_u_tfg<MT, NCLS>(urow, a, m, g, u);
  constexpr int MTI = 3 * MT / 2;  // image blocks per (class, z tile): Cr, Ci - Cr, Cr + Ci
#pragma unroll
  for (int cl = 0; cl < NCLS; ++cl) {
    v4f k1 = v4f{0.f, 0.f, 0.f, 0.f}, k2 = k1, k3 = k1;
#pragma unroll
    for (int qh = 0; qh < MT / 2; ++qh) {
      const float4* zb = lz + ((cl * a.zt + zt) * MTI + qh) * 64 + lane;
      const float4 cr = zb[0], dm = zb[(MT / 2) * 64], sp = zb[MT * 64];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool ok = tfg_index<NCLS>(a, m, g, cl, qh, i) >= 0;
        const float ur = ok ? u[cl][qh][i].x : 0.f, ui = ok ? u[cl][qh][i].y : 0.f;
        k1 = mfma(ur + ui, cr[i], k1);
        k2 = mfma(ur, dm[i], k2);
        k3 = mfma(ui, sp[i], k3);
      }
    }
    Wr[cl] = k1 - k3;
    Wi[cl] = k1 + k2;
  }
  if constexpr (NCLS == 2) {
    const v4f sr = Wr[0] + Wr[1], dr = Wr[0] - Wr[1];
    const v4f si = Wi[0] + Wi[1], di = Wi[0] - Wi[1];
    Wr[0] = sr;
    Wr[1] = dr;
    Wi[0] = si;
    Wi[1] = di;
  }
}

// Even / odd k_t t expansion of one class (E + O at t, E - O at t + 16).
template <int TH>
__device__ __forceinline__ void texp_tfg(const v4f& Wr, const v4f& Wi, const float (&ta)[TH][2][4], float* yb, int m,
                                         int g) {
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
      acc = mfma(ta[mt][0][i], Wr[i], acc);
      acc = mfma(ta[mt][1][i], Wi[i], acc);
    }
#pragma unroll
  for (int mt = 0; mt < TH / 2; ++mt) {
    const int t0 = 16 * mt + 4 * g;
    *reinterpret_cast<v4f*>(yb + yoff(m, t0, 32)) = E[mt] + O[mt];
    *reinterpret_cast<v4f*>(yb + yoff(m, t0 + 16, 32)) = E[mt] - O[mt];
  }
}

// Row g of the result is row 0 (lanes 0..15) of r_g: three gfx950 lane
// swaps (rows of 16 lanes; v_permlane16_swap trades the odd rows of its
// first operand with the even rows of its second, v_permlane32_swap the
// upper half of its first with the lower half of its second).
__device__ __forceinline__ float gather_rows(float r0, float r1, float r2, float r3) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(r0), __float_as_uint(r1), false, false);
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(r2), __float_as_uint(r3), false, false);
  // a[0]: rows r0.0, r1.0, r0.2, r1.2; b[0]: rows r2.0, r3.0, r2.2, r3.2
  const auto c = __builtin_amdgcn_permlane32_swap(a[0], b[0], false, false);
  return __uint_as_float(c[0]);
}

// Sum over the four 16-lane rows of r_g, left in row g (a reduce-scatter of
// the 4 x 4 (row, register) values of each lane position): two
// v_permlane32_swap pairs and one v_permlane16_swap pair with their sums.
__device__ __forceinline__ float sum_rows_to_row(float r0, float r1, float r2, float r3) {
  const auto p02 = __builtin_amdgcn_permlane32_swap(__float_as_uint(r0), __float_as_uint(r2), false, false);
  const auto p13 = __builtin_amdgcn_permlane32_swap(__float_as_uint(r1), __float_as_uint(r3), false, false);
  // lanes 0..31: r0 of rows (0 + 2, 1 + 3); lanes 32..63: r2 of rows (0 + 2, 1 + 3); likewise r1, r3
  const float s02 = __uint_as_float(p02[0]) + __uint_as_float(p02[1]);
  const float s13 = __uint_as_float(p13[0]) + __uint_as_float(p13[1]);
  const auto q = __builtin_amdgcn_permlane16_swap(__float_as_uint(s02), __float_as_uint(s13), false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}

// KI: K steps of 4 input channels (C_in <= 4 KI); OT: tiles of 16 output
// channels per pass (C_out <= 16 OT OH); SPF: float4 of the row's spectrum
// per thread (C_out K_z K_t <= 2 * 64 kBlkWaves SPF); XD: chunks of x loaded
// ahead; OH: passes over the output channels per chunk.  With OH = 2 (C_out
// up to 32) a pipeline unit is one half of a chunk's output channels (16 of
// them), so the LDS buffers hold 16 channels: the two halves of a chunk run
// in consecutive steps on the same x, which is loaded a chunk (two steps)
// ahead into the buffer the previous chunk has released.
//
// The loop is software-pipelined: step c runs phase 2 of chunk c - 1 and
// phase 1 of chunk c (they use different LDS buffers, so the wave's matrix
// products of one overlap the vector work and the memory traffic of the
// other), then one barrier.  Steps come in passes of four so that the
// buffer, the fold class of phase 1 and the x buffer are compile-time indices.
template <int CT, int TH, int MT, int NCLS, int TF, int KI, int OT, int SPF, int XD, int OH>
__global__ void __launch_bounds__(64 * kBlkWaves)
inv_zt_block_kernel(const float2* __restrict__ in, const float* __restrict__ x, const float* __restrict__ wb,
                    float* __restrict__ y, const float* __restrict__ timg, const float4* __restrict__ zimg,
                    StreamArgs a, BlockArgs ba) {
  constexpr int NW = kBlkWaves;
  // output channels per wave in phase 1 (the class bounds C_in and C_out by 4 KI),
  // KCH of them per pass over the output channels
  constexpr int KC = (4 * KI + NW - 1) / NW;
  constexpr int KCH = KC / OH;
  static_assert(OH == 1 || (OH == 2 && OT == 1 && XD == 2 && 16 % NW == 0 && KCH * NW == 16),
                "output halves of 16 channels, x two chunks in flight");
  static_assert(!TF || (CT == 2 && TH == 2), "t folding needs two k_t tiles and N_t = 32");
  static_assert(XD == 1 || XD == 2 || XD == 4, "x one, two or four chunks ahead");
  static_assert(OT == 1 || OT == 2, "one or two output tiles per pass");
  // LDS: the z image, the row's spectrum of every output channel, two
  // buffers of a chunk's expanded values [o][z row][t].
  extern __shared__ float4 lds[];
  const int nimg = NCLS * a.zt * (TF ? 3 * MT / 2 : MT) * 64;  // z image blocks per (class, z tile)
  const int spec_len = a.kz * a.kt;
  const int n4 = ba.co * spec_len / 2;  // float4 of the row's spectrum
  float2* sbuf = reinterpret_cast<float2*>(lds + nimg);
  float* ybuf = reinterpret_cast<float*>(lds + nimg + n4);
  const int bufsz = (OH == 1 ? ba.co : 16) * ba.ostride;  // floats per buffer
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int m = lane & 15, g = lane >> 4;
  const int w = tid >> 6;
  if (blockIdx.x >= ba.rows) return;  // the host never launches more workgroups than rows

  for (int i = tid; i < nimg; i += blockDim.x) lds[i] = zimg[i];

  // A operand of the t expansion (rows t = 16mt + m); with TF only mt < TH/2.
  float ta[TH][CT][4];
#pragma unroll
  for (int mt = 0; mt < TH; ++mt)
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        ta[mt][ct][i] = (TF && mt >= TH / 2) ? 0.f : timg[((mt * CT + ct) * 4 + i) * 64 + lane];
  // A operands of the bypass: w[o = 16ot + m][i = 4s + g], zero outside
  // (row tiles of every pass).
  float wa[OH * OT][KI];
#pragma unroll
  for (int ot = 0; ot < OH * OT; ++ot)
#pragma unroll
    for (int s = 0; s < KI; ++s) {
      const int o = 16 * ot + m, i = 4 * s + g;
      wa[ot][s] = (o < ba.co && i < ba.ci) ? wb[o * ba.ci + i] : 0.f;
    }
  // A class whose full channel count leaves a last tile of 4 channels (C =
  // 20) takes that tile, in its unconditional passes, on the 4 x 4 x 1
  // sixteen-block products (block b = lanes 4b..4b+3: A from lane 4b + i, B
  // from lane 4b + j, D[i][j] in register i of lane 4b + j): A of lane
  // (m, g) is w[o4 + m % 4][4s + g], B its own x of channel 4s + g at point
  // 4m + jj, so register i of lane (m, g) sums the channels 4s + g of output
  // channel o4 + i at point 4m + jj, and a sum over the four rows completes
  // it.  A quarter of the matrix work of a 16-row tile with 12 empty rows.
  constexpr bool kPart4 = OH == 1 && OT > 1 && 16 * (OT - 1) + 4 == 4 * KI;
  constexpr int o4 = 16 * (OT - 1);
  float wp[kPart4 ? KI : 1];
#pragma unroll
  for (int s = 0; s < (kPart4 ? KI : 1); ++s) {
    const int o = o4 + (m & 3), i = 4 * s + g;
    wp[s] = (kPart4 && o < ba.co && i < ba.ci) ? wb[o * ba.ci + i] : 0.f;
  }

  const int64_t row_len = int64_t(a.nz) * a.nt;
  const int nt = a.nt;
  const int cpr = a.zt * NCLS;  // chunks per row

  // Channel stride of x and y (floats).
  const int64_t cs = ba.xy * row_len;

  // Chunk position: row, z tile, class; chunks of a row run z tile by z tile.
  // xb, yb: float offsets of channel 0 of the row (b, x, y) in x and y (rows
  // past the end use the last row, whose x the loads past the end re-read).
  struct Cur {
    int64_t row, xb, yb;
    int zt, hf, oh;
  };
  auto at_row = [&](Cur& c) {
    const int64_t rr = c.row < ba.rows ? c.row : ba.rows - 1;
    const int64_t b = rr / ba.xy, rxy = rr - b * ba.xy;
    c.xb = b * ba.ci * cs + rxy * row_len;
    c.yb = b * ba.co * cs + rxy * row_len;
  };
  // next chunk (output pass 0) and next unit (output pass, then chunk)
  auto next_chunk = [&](Cur c) {
    c.oh = 0;
    if (++c.hf == NCLS) {
      c.hf = 0;
      if (++c.zt == a.zt) {
        c.zt = 0;
        c.row += gridDim.x;
        at_row(c);
      }
    }
    return c;
  };
  auto next = [&](Cur c) {
    if (++c.oh < OH) return c;
    return next_chunk(c);
  };

  // This wave's 64-point group of a chunk: offset of the lane's 4 points
  // within the (N_z x N_t) row, LDS offset within a channel of the buffer,
  // and whether the points exist (a wave past the chunk's groups, or a z row
  // past a ragged last z tile).
  struct Grp {
    int off;
    int loff;
    bool ok;
  };
  const int gpo = w * 64 + 4 * m;
  const int gzr = gpo / nt, gt = gpo - gzr * nt;  // z row and t of the lane's points in a chunk
  const bool gok = w < ba.groups;
  const int gloff = gok ? yoff(gzr, gt, nt) : 0;
  auto group = [&](const Cur& c) {
    Grp q;
    const int zl = c.zt * 16 + gzr;
    q.ok = gok && zl < a.zh;
    q.off = q.ok ? (zl + c.hf * a.zh) * nt + gt : 0;
    q.loff = gloff;
    return q;
  };
  // per-lane channel offsets: input channel 4s + g of x, output channel
  // 16ot + 4g + r of y (the rest is uniform)
  const int64_t gcs_x = g * cs, gcs_y = 4 * g * cs;

  // x of this wave's group, XD chunks ahead (unconditional loads: lanes of
  // missing points read the row start, input channels past C_in read the
  // last one; both are multiplied by zero weights or not stored).
  float4 xv[XD][KI];
  // (FAST: C_in = 4 KI, every input channel exists)
  auto load_x = [&](int k, const Cur& c, auto fastc) __attribute__((always_inline)) {
    constexpr bool FAST = decltype(fastc)::value;
    const Grp q = group(c);
    const float* xr = x + c.xb + q.off;
#pragma unroll
    for (int s = 0; s < KI; ++s) {
      const int64_t co = (FAST || 4 * s + g < ba.ci) ? 4 * s * cs + gcs_x : (ba.ci - 1) * cs;
      xv[k][s] = *reinterpret_cast<const float4*>(xr + co);
    }
  };
  // The spectrum of row r (every output channel) into the LDS buffer: the
  // loads go out first and the LDS stores follow the caller's other work.
  auto spec_load = [&](int64_t r, v4f (&sp)[SPF]) __attribute__((always_inline)) {
    const int64_t rr = r < ba.rows ? r : ba.rows - 1;
    const int64_t b = rr / ba.xy, rxy = rr - b * ba.xy;
#pragma unroll
    for (int k = 0; k < SPF; ++k) {
      const int e4 = min(tid + 64 * NW * k, n4 - 1);
      const int o = (2 * e4) / spec_len, j = 2 * e4 - o * spec_len;
      sp[k] = *reinterpret_cast<const v4f*>(in + ((b * ba.co + o) * ba.xy + rxy) * spec_len + j);
    }
  };
  // (lanes past the end loaded entry n4 - 1 and store that same value to
  // it: no per-lane condition, which the compiler would keep as a scalar
  // lane mask for every k across the whole loop)
  auto spec_store = [&](const v4f (&sp)[SPF]) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < SPF; ++k) reinterpret_cast<v4f*>(sbuf)[min(tid + 64 * NW * k, n4 - 1)] = sp[k];
  };

  // z expansions of this wave's channels, kept for the z tile's chunks
  v4f Wz[KC][NCLS][CT];              // unfolded t
  v4f Wzr[KC][NCLS], Wzi[KC][NCLS];  // t folded

  // Phase 1 of unit c (chunk class HF, output pass OHI) into buffer PAR:
  // this wave's channels o = 16 OHI + w + NW k of the pass (o = w + NW k
  // with one pass), at buffer channel o - 16 OHI.
  auto phase1 = [&](auto parc, auto hfc, auto ohc, auto fastc, const Cur& c) __attribute__((always_inline)) {
    constexpr int PAR = decltype(parc)::value, HF = decltype(hfc)::value, OHI = decltype(ohc)::value;
    constexpr bool FAST = decltype(fastc)::value;
    float* yb = ybuf + PAR * bufsz;
    // (Channel o, slot k of this wave, exists; in the unconditional passes,
    // C_out = 4 KI, this is known at compile time for the slots whose
    // channels all lie below 4 KI.)
#define DTST_BLK_HAS(k, o) ((FAST && 16 * OHI + NW * ((k) + 1) <= 4 * KI) || (o) < ba.co)
    if constexpr (TF) {
#pragma unroll
      for (int k = 0; k < KCH; ++k) {
        const int kk = OHI * KCH + k, ol = w + NW * k, o = 16 * OHI + ol;
        if (DTST_BLK_HAS(k, o)) {
          if (HF == 0) zexp_tfg<MT, NCLS>(sbuf + o * spec_len, a, lds, c.zt, m, g, lane, Wzr[kk], Wzi[kk]);
          texp_tfg<TH>(Wzr[kk][HF], Wzi[kk][HF], ta, yb + ol * ba.ostride, m, g);
        }
      }
    } else {
      if (HF == 0) {
        float4 Bz[NCLS][MT];
#pragma unroll
        for (int cl = 0; cl < NCLS; ++cl)
#pragma unroll
          for (int q = 0; q < MT; ++q) Bz[cl][q] = lds[((cl * a.zt + c.zt) * MT + q) * 64 + lane];
#pragma unroll
        for (int k = 0; k < KCH; ++k) {
          const int kk = OHI * KCH + k, o = 16 * OHI + w + NW * k;
          if (DTST_BLK_HAS(k, o)) zexp_plain<CT, MT, NCLS>(sbuf + o * spec_len, a, Bz, m, g, Wz[kk]);
        }
      }
#pragma unroll
      for (int k = 0; k < KCH; ++k) {
        const int kk = OHI * KCH + k, ol = w + NW * k, o = 16 * OHI + ol;
        // (FAST: N_t = 16 TH, every t row exists)
        if (DTST_BLK_HAS(k, o)) texp_plain<CT, TH, FAST>(Wz[kk][HF], ta, yb + ol * ba.ostride, nt, m, g);
      }
    }
  };

#undef DTST_BLK_HAS

  // Phase 2 of unit c (output pass OHI: channels 16 (OHI OT + ot) + 4g + r,
  // buffer channel 16 ot + 4g + r) from buffer PAR with x buffer XB, in two
  // parts.  The matrix part: the expanded values from LDS plus the bypass
  // products, into C.
  auto phase2_mma = [&](auto parc, auto xbc, auto ohc, auto fastc, const Cur& c, v4f (&C)[OT][4])
                        __attribute__((always_inline)) {
    constexpr int PAR = decltype(parc)::value, XB = decltype(xbc)::value, OHI = decltype(ohc)::value;
    constexpr bool FAST = decltype(fastc)::value;
    const float* yb = ybuf + PAR * bufsz;
    const Grp q = group(c);
#pragma unroll
    for (int ot = 0; ot < OT - (FAST && kPart4 ? 1 : 0); ++ot)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int ol = 16 * ot + 4 * g + r, o = 16 * OHI * OT + ol;
        const bool whole = FAST && 16 * (OHI * OT + ot) + 16 <= 4 * KI;  // tile known to be full
        const float4 v = *reinterpret_cast<const float4*>(yb + (whole || o < ba.co ? ol : 0) * ba.ostride + q.loff);
        C[ot][0][r] = v.x;
        C[ot][1][r] = v.y;
        C[ot][2][r] = v.z;
        C[ot][3][r] = v.w;
      }
    // the 4-channel tile of the unconditional passes (see wp): C[OT - 1][jj]
    // holds its row-partial sums at point 4m + jj, from zero (the expanded
    // values are added after the row sum)
    constexpr bool P4 = FAST && kPart4;
    if constexpr (P4) {
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) C[OT - 1][jj] = v4f{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int s = 0; s < KI; ++s) {
      const bool iok = FAST || 4 * s + g < ba.ci;
      const float4 xs = xv[XB][s];
      const float b0 = iok ? xs.x : 0.f, b1 = iok ? xs.y : 0.f, b2 = iok ? xs.z : 0.f, b3 = iok ? xs.w : 0.f;
#pragma unroll
      for (int ot = 0; ot < OT - (P4 ? 1 : 0); ++ot) {
        const float wv = wa[OHI * OT + ot][s];
        C[ot][0] = mfma(wv, b0, C[ot][0]);
        C[ot][1] = mfma(wv, b1, C[ot][1]);
        C[ot][2] = mfma(wv, b2, C[ot][2]);
        C[ot][3] = mfma(wv, b3, C[ot][3]);
      }
      if constexpr (P4) {
        C[OT - 1][0] = __builtin_amdgcn_mfma_f32_4x4x1f32(wp[s], b0, C[OT - 1][0], 0, 0, 0);
        C[OT - 1][1] = __builtin_amdgcn_mfma_f32_4x4x1f32(wp[s], b1, C[OT - 1][1], 0, 0, 0);
        C[OT - 1][2] = __builtin_amdgcn_mfma_f32_4x4x1f32(wp[s], b2, C[OT - 1][2], 0, 0, 0);
        C[OT - 1][3] = __builtin_amdgcn_mfma_f32_4x4x1f32(wp[s], b3, C[OT - 1][3], 0, 0, 0);
      }
    }
  };
  // The vector part in the unconditional passes (C_out = 4 KI, every point
  // present): GELU and stores without conditions (a last tile of 4 channels
  // gathered across rows).
  auto phase2_store_full = [&](auto parc, auto ohc, const Cur& c, const v4f (&C)[OT][4])
                               __attribute__((always_inline)) {
    constexpr int PAR = decltype(parc)::value, OHI = decltype(ohc)::value;
    const Grp q = group(c);
    const int off = q.off;
    float* yr = y + c.yb + gcs_y + off;
    auto tile = [&](auto otc) __attribute__((always_inline)) {
      constexpr int ot = decltype(otc)::value, o0 = 16 * (OHI * OT + ot);
      if constexpr (o0 + 16 <= 4 * KI) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          *reinterpret_cast<v4f*>(yr + (o0 + r) * cs) =
              v4f{gelu_as(C[ot][0][r]), gelu_as(C[ot][1][r]), gelu_as(C[ot][2][r]), gelu_as(C[ot][3][r])};
      } else if constexpr (kPart4) {
        static_assert(o0 == o4 && o0 + 4 == 4 * KI, "the 4-channel tile is the last one");
        // row g: output channel o0 + g at the lane's points 4m..4m+3, plus the
        // expanded values of that channel
        const float4 e = *reinterpret_cast<const float4*>(ybuf + PAR * bufsz + (16 * ot + g) * ba.ostride + q.loff);
        const float e4[4] = {e.x, e.y, e.z, e.w};
        float v[4];
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
          v[jj] = gelu_as(sum_rows_to_row(C[ot][jj][0], C[ot][jj][1], C[ot][jj][2], C[ot][jj][3]) + e4[jj]);
        *reinterpret_cast<v4f*>(y + c.yb + int64_t(o0 + g) * cs + off) = v4f{v[0], v[1], v[2], v[3]};
      } else {
        static_assert(o0 + 4 == 4 * KI, "a partial tile of the unconditional passes has 4 channels");
        float* yc = y + c.yb + int64_t(o0) * cs + off + g;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          yc[r * cs] = gelu_as(gather_rows(C[ot][0][r], C[ot][1][r], C[ot][2][r], C[ot][3][r]));
      }
    };
    tile(std::integral_constant<int, 0>{});
    if constexpr (OT > 1) tile(std::integral_constant<int, 1>{});
  };
  // The whole of phase 2 with every condition (ragged tiles, missing points
  // and channels).
  auto phase2 = [&](auto parc, auto xbc, auto ohc, const Cur& c) __attribute__((always_inline)) {
    constexpr int OHI = decltype(ohc)::value;
    const Grp q = group(c);
    v4f C[OT][4];
    phase2_mma(parc, xbc, ohc, std::integral_constant<bool, false>{}, c, C);
    float* yr = y + c.yb + gcs_y + q.off;
#pragma unroll
    for (int ot = 0; ot < OT; ++ot) {
      const int o0 = 16 * (OHI * OT + ot);  // first output channel of the tile
      if (ba.co - o0 <= 4) {
        // At most 4 channels (C_out = 20 of the paper's width, say): only the
        // lanes g = 0 hold outputs.  Lane (m, g) takes point 4m + g of lane
        // (m, 0) for each of the 4 channels, so that every lane evaluates 4
        // GELUs instead of the 16 of a full tile; each store then covers the
        // group's 64 points of one channel (256 bytes).
        if (ba.co > o0) {
          float* yc = y + c.yb + int64_t(o0) * cs + q.off + g;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float v = gather_rows(C[ot][0][r], C[ot][1][r], C[ot][2][r], C[ot][3][r]);
            if (q.ok && o0 + r < ba.co) yc[r * cs] = gelu_as(v);
          }
        }
        continue;
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int o = o0 + 4 * g + r;
        if (q.ok && o < ba.co) {
          float* dst = yr + (o0 + r) * cs;
          // ordinary (cached) stores: measured faster here than streaming ones
          *reinterpret_cast<v4f*>(dst) =
              v4f{gelu_as(C[ot][0][r]), gelu_as(C[ot][1][r]), gelu_as(C[ot][2][r]), gelu_as(C[ot][3][r])};
        }
      }
    }
  };

  // One pipeline step: phase 2 of chunk c2 (the previous one, when it
  // exists), the x of the chunk XD - 1 further on into phase 2's x buffer,
  // phase 1 of chunk c1 (when it exists), one barrier.  The x loads are
  // unconditional (past the end they re-read the last row), so that no
  // register holding a load in flight is merged with another value.  The
  // step whose phase 1 is a row's last chunk then moves the next row's
  // spectrum into LDS (the row's last reader of it is the phase 1 of its last
  // z tile's first chunk).
  Cur c1 = Cur{static_cast<int64_t>(blockIdx.x), 0, 0, 0, 0, 0};  // phase 1
  at_row(c1);
  Cur c2 = c1;                                             // phase 2 (valid from step 1 on)
  Cur cx = c1;                                             // next x to load
  auto step = [&](auto sc, auto fastc, bool has2) __attribute__((always_inline)) {
    constexpr bool FAST = decltype(fastc)::value;
    constexpr int S4 = decltype(sc)::value;     // step index mod 4
    constexpr int PAR = S4 & 1;                 // buffer of phase 1; phase 2 reads 1 - PAR
    // output pass of phase 1's unit and of phase 2's (the previous) unit
    constexpr int OH1 = OH == 2 ? (S4 & 1) : 0, OH2 = OH == 2 ? 1 - OH1 : 0;
    // class of phase 1's chunk: chunks alternate classes when z folds
    constexpr int HF = NCLS == 2 ? (OH == 2 ? (S4 >> 1) & 1 : PAR) : 0;
    // x buffer of phase 2's chunk: the previous step's chunk with one pass;
    // with two passes unit u - 1 belongs to chunk (u - 1) / 2 (buffers by
    // chunk parity: 1, 0, 0, 1 for S4 = 0..3), and the odd steps (phase 2
    // on a chunk's first pass) load the next chunk into the other buffer,
    // which the previous chunk released at the step before
    constexpr int XB = OH == 2 ? ((S4 == 0 || S4 == 3) ? 1 : 0) : (S4 + 3) % XD;
    constexpr int XL = OH == 2 ? 1 - XB : XB;
    constexpr bool LOADS = OH == 1 || (S4 & 1) == 1;
    const bool has1 = FAST || c1.row < ba.rows;
    auto body = [&]() __attribute__((always_inline)) {
      using P1 = std::integral_constant<int, PAR>;
      using P2 = std::integral_constant<int, 1 - PAR>;
      if constexpr (FAST) {
        // Both phases unconditional: the step is one basic block (no
        // per-channel or per-store branches), which the compiler schedules
        // as a whole.  (Taking the two phases in opposite orders on the two
        // waves of a SIMD was measured slower: C held across phase 1 spills.)
        v4f C[OT][4];
        phase2_mma(P2{}, std::integral_constant<int, XB>{}, std::integral_constant<int, OH2>{}, fastc, c2, C);
        if constexpr (LOADS) {
          load_x(XL, cx, fastc);
          cx = next_chunk(cx);
        }
        phase2_store_full(P2{}, std::integral_constant<int, OH2>{}, c2, C);
        phase1(P1{}, std::integral_constant<int, HF>{}, std::integral_constant<int, OH1>{}, fastc, c1);
      } else {
        if (has2)
          phase2(P2{}, std::integral_constant<int, XB>{}, std::integral_constant<int, OH2>{}, c2);
        if constexpr (LOADS) {
          load_x(XL, cx, fastc);
          cx = next_chunk(cx);
        }
        if (has1) phase1(P1{}, std::integral_constant<int, HF>{}, std::integral_constant<int, OH1>{}, fastc, c1);
      }
    };
    // (c1.hf == HF and c1.oh == OH1 by construction: only the steps whose
    // unit is the last class and pass of a chunk can end a row)
    if (has1 && HF == NCLS - 1 && OH1 == OH - 1 && c1.zt == a.zt - 1) {
      // the spectrum loads go out before the step's work, the LDS stores after it
      v4f sp[SPF];
      spec_load(c1.row + gridDim.x, sp);
      body();
      if constexpr (NCLS == 1) __syncthreads();  // this phase 1 read the spectrum buffer (z expansion)
      spec_store(sp);
    } else {
      body();
    }
    __syncthreads();
    c2 = c1;
    c1 = next(c1);
  };

  // prologue: the first row's spectrum, the x of the first XD - 1 chunks
  {
    v4f sp[SPF];
    spec_load(c1.row, sp);
    spec_store(sp);
  }
#pragma unroll
  for (int k = 0; k < XD - 1; ++k) {
    load_x(k, cx, std::integral_constant<bool, false>{});
    cx = next_chunk(cx);
  }
  __syncthreads();
  using Gen = std::integral_constant<bool, false>;
  using Fast = std::integral_constant<bool, true>;
  step(std::integral_constant<int, 0>{}, Gen{}, false);
  // Passes whose four units all exist run the unconditional steps when the
  // channel counts fill the class (C_in = C_out = 4 KI: 16, 20 or 32, the
  // last tile of 20 with 4 channels) and every chunk is complete (N_t = 4 NW,
  // whole z tiles).
  constexpr bool kFull = 16 * OT * OH == 4 * KI || (OH == 1 && 16 * (OT - 1) + 4 == 4 * KI);
  const bool full = kFull && ba.co == 4 * KI && ba.ci == 4 * KI && nt == 4 * NW && a.zh % 16 == 0;
  const int64_t units = ((ba.rows - 1 - blockIdx.x) / gridDim.x + 1) * cpr * OH;  // this workgroup's units
  int64_t u1 = 1;  // unit of c1
  // Every pass runs four steps; the only exits are at the end of a pass.
  // The unconditional passes come first (they are contiguous), in a loop of
  // their own, so that the loop-invariant values of the other steps (lane
  // masks of their conditions, among others) are not held across them.
  if constexpr (kFull) {
    if (full) {
      while (u1 + 3 < units) {
        step(std::integral_constant<int, 1>{}, Fast{}, true);
        step(std::integral_constant<int, 2>{}, Fast{}, true);
        step(std::integral_constant<int, 3>{}, Fast{}, true);
        step(std::integral_constant<int, 0>{}, Fast{}, true);
        u1 += 4;
      }
    }
  }
  // (c2 holds a unit that exists after step 0 and after any unconditional
  // pass, so this loop runs at least once)
  while (c2.row < ba.rows) {
    step(std::integral_constant<int, 1>{}, Gen{}, c2.row < ba.rows);
    step(std::integral_constant<int, 2>{}, Gen{}, c2.row < ba.rows);
    step(std::integral_constant<int, 3>{}, Gen{}, c2.row < ba.rows);
    step(std::integral_constant<int, 0>{}, Gen{}, c2.row < ba.rows);
  }
}

typedef void (*blk_fn)(const float2*, const float*, const float*, float*, const float*, const float4*, StreamArgs,
                       BlockArgs);

template <int CT, int TH, int MT, int NCLS, int TF>
blk_fn pick_kio(int kio) {
  if (kio == 0) return inv_zt_block_kernel<CT, TH, MT, NCLS, TF, 4, 1, 4, 2, 1>;
  if (kio == 1) return inv_zt_block_kernel<CT, TH, MT, NCLS, TF, 5, 2, 5, 1, 1>;
  return inv_zt_block_kernel<CT, TH, MT, NCLS, TF, 8, 1, 8, 2, 2>;
}

// float4 of a row's spectrum per thread for each (KI, OT) class.
constexpr int kSpf[3] = {4, 5, 8};

template <int CT, int TH, int TF>
blk_fn pick_mn(int mt, int ncls, int kio) {
  if (mt == 2) return ncls == 2 ? pick_kio<CT, TH, 2, 2, TF>(kio) : pick_kio<CT, TH, 2, 1, TF>(kio);
  return ncls == 2 ? pick_kio<CT, TH, 4, 2, TF>(kio) : pick_kio<CT, TH, 4, 1, TF>(kio);
}

// (KI, OT) class of a channel count: 0 up to 16, 1 up to 20, 2 up to 32.
int kio_of(int64_t ci, int64_t co) {
  const int64_t c = ci > co ? ci : co;
  return c <= 16 ? 0 : (c <= 20 ? 1 : 2);
}

blk_fn pick_blk(const StreamCfg& c, int kio) {
  if (c.tf) return pick_mn<2, 2, 1>(c.mt, c.ncls, kio);
  if (c.ct == 1) return c.th == 1 ? pick_mn<1, 1, 0>(c.mt, c.ncls, kio) : pick_mn<1, 2, 0>(c.mt, c.ncls, kio);
  return c.th == 1 ? pick_mn<2, 1, 0>(c.mt, c.ncls, kio) : pick_mn<2, 2, 0>(c.mt, c.ncls, kio);
}

}  // namespace

size_t block_zt_lds_bytes(const StreamCfg& c, int64_t ci, int64_t co) {
  // chunk buffers of 16 channels where the instance makes two output passes
  const int64_t cb = kio_of(ci, co) == 2 ? 16 : co;
  return size_t(c.ncls) * c.zt * (c.tf ? 3 * c.mt / 2 : c.mt) * 64 * 16 + size_t(co) * c.kz * c.kt * 8 +
         2 * size_t(cb) * 16 * c.nt * sizeof(float);
}

bool block_zt_supported(const StreamCfg& c, int64_t ci, int64_t co) {
  if (!(c.vec && c.th <= 2 && c.ncls <= 2 && (c.mt == 2 || c.mt == 4) && (!c.tf || (c.ct == 2 && c.th == 2)) &&
        ci <= 32 && co <= 32 && (c.kz * c.kt) % 2 == 0))
    return false;
  const int64_t n4 = co * c.kz * c.kt / 2;
  return n4 <= int64_t(64) * kBlkWaves * kSpf[kio_of(ci, co)] && block_zt_lds_bytes(c, ci, co) <= 160 * 1024;
}

int prepare_block_zt(const StreamCfg& c, int64_t ci, int64_t co, int* grid) {
  const void* fn = reinterpret_cast<const void*>(pick_blk(c, kio_of(ci, co)));
  const size_t lds = block_zt_lds_bytes(c, ci, co);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  if (e != hipSuccess) return e;
  int dev = 0, cus = 0, per_cu = 0;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 64 * kBlkWaves, lds)) != hipSuccess) return e;
  if (per_cu <= 0) return hipErrorInvalidConfiguration;
  *grid = cus * per_cu;
  return hipSuccess;
}

int launch_inv_zt_block(const StreamCfg& c, int grid_resident, const void* in, const float* x, const float* w,
                        float* y, int64_t batch, int64_t nxy, int64_t ci, int64_t co, const float* timg,
                        const float* zimg, void* stream) {
  const int64_t rows = batch * nxy;
  if (rows <= 0) return hipSuccess;
  if (!block_zt_supported(c, ci, co) || grid_resident <= 0) return hipErrorInvalidConfiguration;
  StreamArgs a;
  a.rows = rows;
  a.nt = c.nt;
  a.nz = c.nz;
  a.kt = c.kt;
  a.kz = c.kz;
  a.zh = c.zh;
  a.zt = c.zt;
  a.vec = c.vec;
  a.full = 0;
  BlockArgs ba;
  ba.rows = rows;
  ba.xy = nxy;
  ba.ci = static_cast<int>(ci);
  ba.co = static_cast<int>(co);
  ba.groups = c.nt / 4;
  ba.ostride = 16 * c.nt;
  if (ba.groups > kBlkWaves) return hipErrorInvalidConfiguration;
  const int64_t grid = rows < grid_resident ? rows : grid_resident;
  hipLaunchKernelGGL(pick_blk(c, kio_of(ci, co)), dim3(static_cast<unsigned>(grid)), dim3(64 * kBlkWaves),
                     block_zt_lds_bytes(c, ci, co), static_cast<hipStream_t>(stream), static_cast<const float2*>(in), x,
                     w, y, timg, reinterpret_cast<const float4*>(zimg), a, ba);
  return hipGetLastError();
}

}  // namespace dtst
