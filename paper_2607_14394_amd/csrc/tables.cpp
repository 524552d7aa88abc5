// Host-side geometry validation and basis tables of the DTST library.
//
// Everything here is plain C++ (no HIP): it derives the kernel
// configuration from a descriptor and builds, in fp64, the kernel-ready
// images of the per-dimension basis matrices of Sec. V-B Eq. (basis_matrix),
//   B_i[k, j] = exp(-2 pi i ((k * (offset_i + j)) mod N_i) / N_i),
// each value rounded once to fp32.  The exponent is reduced in exact
// integer arithmetic before the angle is formed, so no precision is lost to
// large k*n products (k*n reaches 2.6e5 at N = 512).
#include <algorithm>
#include <cmath>
#include <limits>

#include "dtst_internal.h"

namespace dtst {

namespace {

constexpr double kTwoPi = 6.283185307179586476925286766559;

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t round_up(size_t a, size_t b) { return (a + b - 1) / b * b; }

// exp(-2 pi i r / N) with r = (k * n) mod N, k, n >= 0.
inline void twiddle(int64_t N, int64_t k, int64_t n, double* re, double* im) {
  const int64_t r = ((k % N) * (n % N)) % N;
  const double ang = kTwoPi * static_cast<double>(r) / static_cast<double>(N);
  *re = std::cos(ang);
  *im = -std::sin(ang);
}

// Real-inverse weight of stored t index kt (Sec. V-A inverse, half spectrum).
inline double half_weight(int64_t nt, int64_t kt) {
  if (kt == 0) return 1.0;
  if (nt % 2 == 0 && kt == nt / 2) return 1.0;
  return 2.0;
}

// Classes stacked in an inverse axis image entry (fold 2: parity, fold 4:
// k mod 4); the forward images hold one class per k tile.
inline int axis_image_classes(const AxisCfg& a) { return a.fold == 2 ? 2 : (a.fold == 4 ? 4 : 1); }

// z image blocks of 16 rows (forward) or 16 K entries (inverse) per (class,
// z tile): mt, plus mt / 2 when t folds (the three-product form's third
// operand, see z_forward_image and z_inverse_image).
inline int z_blocks(const StreamCfg& s) { return s.tf ? 3 * s.mt / 2 : s.mt; }

bool mul_ok(int64_t a, int64_t b, int64_t* out) {
  if (a < 0 || b < 0) return false;
  if (a != 0 && b > std::numeric_limits<int64_t>::max() / a) return false;
  *out = a * b;
  return true;
}

}  // namespace

int64_t retained_index(const dtst_desc& d, int dim, int64_t p) {
  if (dim == 3) return p;
  const int64_t k = d.kmax[dim];
  return p < k ? p : d.n_global[dim] - 2 * k + p;
}

dtst_status derive(const dtst_desc* d, uint32_t flags, Derived* out, std::string* err) {
  if (!d || !out) {
    *err = "null descriptor";
    return DTST_ERR_INVALID_ARG;
  }
  static const char* names[4] = {"x", "y", "z", "t"};
  for (int i = 0; i < 4; ++i) {
    if (d->n_global[i] < 1 || d->n_local[i] < 1 || d->offset[i] < 0 ||
        d->n_local[i] > d->n_global[i] || d->offset[i] > d->n_global[i] - d->n_local[i]) {
      *err = std::string("dimension ") + names[i] +
             ": need n_global >= 1, n_local >= 1, 0 <= offset, offset + n_local <= n_global";
      return DTST_ERR_INVALID_ARG;
    }
    if (d->n_global[i] > (int64_t(1) << 30)) {
      *err = std::string("dimension ") + names[i] + ": n_global above 2^30";
      return DTST_ERR_INVALID_ARG;
    }
  }
  for (int i = 0; i < 3; ++i) {
    if (d->kmax[i] < 1 || 2 * int64_t(d->kmax[i]) > d->n_global[i]) {
      *err = std::string("dimension ") + names[i] + ": need 1 <= 2*kmax <= n_global";
      return DTST_ERR_INVALID_ARG;
    }
  }
  if (d->kt < 1 || d->kt > d->n_global[3] / 2 + 1) {
    *err = "t: need 1 <= kt <= n_global_t/2 + 1";
    return DTST_ERR_INVALID_ARG;
  }
  if (d->batch < 0 || d->c_in < 1 || d->c_out < 1) {
    *err = "need batch >= 0, c_in >= 1, c_out >= 1";
    return DTST_ERR_INVALID_ARG;
  }
  if ((flags & ~uint32_t(DTST_PLAN_SPLIT_SCHEDULE | DTST_PLAN_UNFUSED_BLOCK)) != 0) {
    *err = "unknown plan flag";
    return DTST_ERR_INVALID_ARG;
  }

  Derived dv;
  dv.d = *d;
  for (int i = 0; i < 3; ++i) dv.K[i] = 2 * int64_t(d->kmax[i]);
  dv.K[3] = d->kt;
  dv.M = dv.K[0] * dv.K[1] * dv.K[2] * dv.K[3];

  // Element counts must stay far inside int64.
  const int64_t cmax = std::max(d->c_in, d->c_out);
  int64_t t = 1;
  bool ok = mul_ok(std::max<int64_t>(d->batch, 1), cmax, &t);
  for (int i = 0; i < 4 && ok; ++i) ok = mul_ok(t, d->n_local[i], &t);
  int64_t tm = 1;
  ok = ok && mul_ok(std::max<int64_t>(d->batch, 1), cmax, &tm) && mul_ok(tm, dv.M, &tm);
  int64_t tw = 1;
  ok = ok && mul_ok(dv.M, d->c_in, &tw) && mul_ok(tw, d->c_out, &tw);
  if (!ok || t > (int64_t(1) << 50) || tm > (int64_t(1) << 50) || tw > (int64_t(1) << 50)) {
    *err = "problem size overflows the supported element counts";
    return DTST_ERR_INVALID_ARG;
  }

  // ---- streaming t+z configuration ----
  StreamCfg& sc = dv.sc;
  sc.nt = static_cast<int>(d->n_local[3]);
  sc.nz = static_cast<int>(d->n_local[2]);
  sc.kt = d->kt;
  sc.kz = static_cast<int>(dv.K[2]);
  if (sc.kt <= 8) {
    sc.ct = 1;
  } else if (sc.kt <= 16) {
    sc.ct = 2;
  } else {
    *err = "kt > 16 is not covered by the streaming kernels";
    return DTST_ERR_UNSUPPORTED;
  }
  if (sc.nt <= 16) {
    sc.th = 1;
  } else if (sc.nt <= 32) {
    sc.th = 2;
  } else if (sc.nt <= 64) {
    sc.th = 4;
  } else {
    *err = "local N_t > 64 is not covered by the streaming kernels";
    return DTST_ERR_UNSUPPORTED;
  }
  // z folds when this shard holds the whole even z extent: into 2 classes by
  // mode parity, or into 4 by k mod 4 when N_z % 4 == 0 and the stored
  // position of a mode has its residue (k even).  The four-class fold takes
  // either Re / Im of k_t in separate column tiles (ct == 2, the factors +-i
  // swap tiles) with at most 16 modes per class (one Re and one Im row tile:
  // the kernels fit their registers only at that size), or one column tile
  // (ct == 1, the factors +-i trade lanes m and m ^ 8) with at most 8 modes
  // per class, whose Re and Im rows then share one 16-row tile (mt == 1).
  // The z products per row are (padded slots per class) x N_z whatever the
  // class count, so the count taken is the one with the fewest padded slots
  // per class, and of those the smallest (fewer class sums and differences):
  // with at most 16 modes every count pads to one 16-row tile.
  const bool fold = d->n_local[2] == d->n_global[2] && d->n_global[2] % 2 == 0;
  const bool fold4_base = fold && d->n_global[2] % 4 == 0 && d->kmax[2] % 2 == 0;
  const bool fold4_ct2 = fold4_base && sc.ct == 2 && sc.kz <= 4 * 16;
  const bool fold4_ct1 = fold4_base && sc.ct == 1 && sc.kz <= 4 * 8;
  auto padded = [&](int n) {
    if (n == 4 && sc.ct == 1) return 8;
    int k = static_cast<int>(round_up(ceil_div(sc.kz, n), 16));
    return k == 48 ? 64 : k;
  };
  sc.ncls = 1;
  if (fold && padded(2) < padded(sc.ncls)) sc.ncls = 2;
  if ((fold4_ct2 || fold4_ct1) && padded(4) < padded(sc.ncls)) sc.ncls = 4;
  int kcp = padded(sc.ncls);
  if (kcp > 64) {
    *err = "more than 64 retained z modes per parity class is not covered";
    return DTST_ERR_UNSUPPORTED;
  }
  sc.kcp = kcp;
  sc.mt = kcp / 8;
  sc.zh = sc.nz / sc.ncls;
  sc.zt = static_cast<int>(ceil_div(sc.zh, 16));
  sc.vec = (sc.nt % 4 == 0) ? 1 : 0;
  // t folds (even k_t from x(t) + x(t + N_t/2), odd k_t from the difference)
  // in the split kernels when the shard holds the whole t extent of 32.
  sc.tf = (sc.ct == 2 && sc.th == 2 && sc.nt == 32 && d->n_local[3] == d->n_global[3]) ? 1 : 0;
  sc.lds_bytes = size_t(sc.ncls) * sc.zt * z_blocks(sc) * 64 * 16;
  if (sc.lds_bytes > 160 * 1024) {
    *err = "z basis image exceeds the 160 KiB LDS of a workgroup";
    return DTST_ERR_UNSUPPORTED;
  }

  // ---- axis contractions ----
  auto axis = [](int J, int KO, int64_t NN, int fold) {
    AxisCfg a;
    a.J = J;
    a.KO = KO;
    a.NN = static_cast<int>(NN);
    a.fold = fold;
    if (fold == 1) {
      a.JQ = static_cast<int>(ceil_div(J / 2, 16));
      a.kth = static_cast<int>(ceil_div(KO / 2, 16));
      a.ktiles = 2 * a.kth;
    } else if (fold == 2) {
      a.JQ = static_cast<int>(ceil_div(J / 2, 16));
      a.ktiles = static_cast<int>(ceil_div(KO / 2, 16));
    } else if (fold == 3) {
      a.JQ = static_cast<int>(ceil_div(J / 4, 16));
      a.kth = static_cast<int>(ceil_div(KO / 4, 16));
      a.ktiles = 4 * a.kth;
    } else if (fold == 4) {
      a.JQ = static_cast<int>(ceil_div(J / 4, 16));
      a.ktiles = static_cast<int>(ceil_div(KO / 4, 16));
    } else {
      a.JQ = static_cast<int>(ceil_div(J, 16));
      a.ktiles = static_cast<int>(ceil_div(KO, 16));
    }
    return a;
  };
  const int64_t nn_y = dv.K[2] * dv.K[3];
  const int64_t nn_x = dv.K[1] * nn_y;
  if (nn_x > (int64_t(1) << 30)) {
    *err = "retained mode count too large";
    return DTST_ERR_UNSUPPORTED;
  }
  // A dimension folds when this shard holds its whole even global extent.
  const bool fold_x = d->n_local[0] == d->n_global[0] && d->n_global[0] % 2 == 0;
  const bool fold_y = d->n_local[1] == d->n_global[1] && d->n_global[1] % 2 == 0;
  dv.ay_f = axis(static_cast<int>(d->n_local[1]), static_cast<int>(dv.K[1]), nn_y, fold_y ? 1 : 0);
  dv.ax_f = axis(static_cast<int>(d->n_local[0]), static_cast<int>(dv.K[0]), nn_x, fold_x ? 1 : 0);
  dv.ax_i = axis(static_cast<int>(dv.K[0]), static_cast<int>(d->n_local[0]), nn_x, fold_x ? 2 : 0);
  dv.ay_i = axis(static_cast<int>(dv.K[1]), static_cast<int>(d->n_local[1]), nn_y, fold_y ? 2 : 0);

  // ---- workspace: the complex intermediates of the largest channel count ----
  // W1 = (.., N_x, N_y, K_z, K_t) between the t+z and y steps, W2 = (.., N_x,
  // K_y, K_z, K_t) between the y and x steps (W1 only without the fused y).
  const int64_t bc = d->batch * cmax;
  const size_t w1 = round_up(size_t(bc) * d->n_local[0] * d->n_local[1] * nn_y * 8, 256);
  const size_t w2 = round_up(size_t(bc) * d->n_local[0] * dv.K[1] * nn_y * 8, 256);

  // ---- fused forward t + z + y ----
  // Taken when the y contraction fits the fused kernel's registers (one
  // 16-column tile of K_z K_t per wave of 16, at most two 16-row k tiles of
  // K_y per wave) and its LDS.  The plan flag DTST_PLAN_SPLIT_SCHEDULE keeps
  // the separate t + z and y launches.
  {
    const bool split = (flags & DTST_PLAN_SPLIT_SCHEDULE) != 0;
    sc.ncy = fold_y ? 2 : 1;
    sc.kyt = fold_y ? dv.ay_f.kth : dv.ay_f.ktiles;
    const int mcols = static_cast<int>(nn_y);
    sc.fused_mrow = static_cast<int>(round_up(mcols, 32)) + 16;
    // z image, the 16 slots' exchanged rows, and the larger of the forward and
    // inverse y images when that still fits (else the y images are read from
    // global memory)
    const size_t yf = size_t(dv.ay_f.ktiles) * dv.ay_f.JQ * 2 * 64 * 16;
    const size_t yi = size_t(dv.ay_i.ktiles) * dv.ay_i.JQ * (fold_y ? 2 : 1) * 2 * 64 * 16;
    sc.fused_lds_bytes = sc.lds_bytes + size_t(16) * sc.ncy * sc.fused_mrow * 8;
    sc.fused_y_lds = sc.fused_lds_bytes + std::max(yf, yi) <= 160 * 1024 ? 1 : 0;
    if (sc.fused_y_lds) sc.fused_lds_bytes += std::max(yf, yi);
    sc.fuse_y = (!split && sc.ct == 1 && ((sc.mt == 2 && sc.ncls <= 2) || (sc.mt == 1 && sc.ncls == 4)) &&
                 sc.th <= 2 && sc.vec && dv.K[1] <= 32 &&
                 mcols <= 256 && sc.kyt <= (fold_y ? 1 : 2) && sc.fused_lds_bytes <= 160 * 1024)
                    ? 1
                    : 0;
  }
  dv.w1_bytes = sc.fuse_y ? 0 : w1;
  dv.ws_bytes = dv.w1_bytes + w2;

  // Separate x and y launches fold in four classes (k mod 4, which is the
  // position mod 4 when N % 4 == 0 and k_max is even) when every class fills
  // whole 16-mode tiles (K % 64 == 0) and the inverse's class sums take at
  // most two K steps (K <= 128): a quarter of the direct MFMA work instead of
  // a half.
  {
    auto four = [&](int dim) {
      const int64_t n = d->n_global[dim], k = dv.K[dim];
      return d->n_local[dim] == n && n % 4 == 0 && k % 64 == 0 && k <= 128;
    };
    if (four(1) && !sc.fuse_y) {
      dv.ay_f = axis(static_cast<int>(d->n_local[1]), static_cast<int>(dv.K[1]), nn_y, 3);
      dv.ay_i = axis(static_cast<int>(dv.K[1]), static_cast<int>(d->n_local[1]), nn_y, 4);
    }
    if (four(0)) {
      dv.ax_f = axis(static_cast<int>(d->n_local[0]), static_cast<int>(dv.K[0]), nn_x, 3);
      dv.ax_i = axis(static_cast<int>(dv.K[0]), static_cast<int>(d->n_local[0]), nn_x, 4);
    }
  }

  // Two-part (Re, Im) images: the inverse expansions of the expand kernel
  // (fold 2 or 4 within two K steps) and the y images the fused stream
  // kernels read; dtst_inverse_block expands y with the axis kernels even
  // where the plan fuses y into the stream kernels.
  auto expand_parts = [](AxisCfg& a) {
    if ((a.fold == 2 || a.fold == 4) && a.JQ <= 2) a.parts = 2;
  };
  expand_parts(dv.ax_i);
  expand_parts(dv.ay_i);
  dv.ay_b = dv.ay_i;
  if (sc.fuse_y) dv.ay_f.parts = dv.ay_i.parts = 2;

  // ---- fused inverse z + t expansion and block epilogue ----
  // The same z + t expansion as the split inverse, with z folded into at
  // most two classes (a chunk of the kernel is one z tile of every class),
  // fed by the separate y expansion: dtst_inverse_block's workspace holds W1
  // then W2 even where the layer's own calls fuse y.  The plan flag
  // DTST_PLAN_UNFUSED_BLOCK keeps the inverse and the epilogue separate.
  {
    StreamCfg sb = sc;
    sb.ncls = fold && round_up(ceil_div(sc.kz, 2), 16) < round_up(sc.kz, 16) ? 2 : 1;
    sb.kcp = static_cast<int>(round_up(ceil_div(sc.kz, sb.ncls), 16));
    sb.mt = sb.kcp / 8;
    sb.zh = sb.nz / sb.ncls;
    sb.zt = static_cast<int>(ceil_div(sb.zh, 16));
    sb.lds_bytes = size_t(sb.ncls) * sb.zt * z_blocks(sb) * 64 * 16;
    sb.fuse_y = 0;
    dv.sb = sb;
    dv.blk = ((flags & DTST_PLAN_UNFUSED_BLOCK) == 0 && sb.kcp <= 32 &&
              block_zt_supported(sb, d->c_in, d->c_out))
                 ? 1
                 : 0;
    dv.blk_w1_bytes = dv.blk ? w1 : dv.w1_bytes;
    dv.blk_ws_bytes = dv.blk ? w1 + w2 : dv.ws_bytes;
  }


  // ---- image offsets (floats, 256-byte aligned) ----
  Images& im = dv.img;
  size_t off = 0;
  auto take = [&off](size_t n) {
    size_t o = off;
    off = round_up(off + n, 64);
    return o;
  };
  const size_t t_img = size_t(sc.th) * 4 * sc.ct * 64;
  const size_t z_img = size_t(sc.ncls) * sc.zt * z_blocks(sc) * 64 * 4;
  im.t_fwd = take(t_img);
  im.t_fwd_adjoint_of_inverse = take(t_img);
  im.z_fwd = take(z_img);
  im.t_inv = take(t_img);
  im.t_inv_adjoint_of_forward = take(t_img);
  im.z_inv = take(z_img);
  auto axis_img = [](const AxisCfg& a) {
    return size_t(a.ktiles) * a.JQ * axis_image_classes(a) * a.parts * 64 * 4;
  };
  im.y_fwd = take(axis_img(dv.ay_f));
  im.x_fwd = take(axis_img(dv.ax_f));
  im.y_inv = take(axis_img(dv.ay_i));
  im.x_inv = take(axis_img(dv.ax_i));
  im.y_blk = sc.fuse_y ? take(axis_img(dv.ay_b)) : im.y_inv;
  im.z_blk = take(size_t(dv.sb.ncls) * dv.sb.zt * z_blocks(dv.sb) * 64 * 4);
  im.t_blk = take(t_img);
  im.total = off;

  *out = dv;
  return DTST_OK;
}

namespace {

// Complex basis value of dimension dim at (mode position p, local index j).
inline void bval(const dtst_desc& d, int dim, int64_t p, int64_t j, double* re, double* im) {
  twiddle(d.n_global[dim], retained_index(d, dim, p), d.offset[dim] + j, re, im);
}

// t image of the forward streaming kernel (B operand of the first MFMA):
// entry ((h*4 + j)*CT + ct)*64 + lane holds Bt'[t][c] with t = 16h + 4g + j,
// c = 16ct + m (m = lane & 15, g = lane >> 4); c < 8CT is Re B_t[kt=c][t],
// otherwise Im B_t[kt = c - 8CT][t]; times scale(kt).  t-folded (tf), only
// t < N_t/2 is filled and column m of tile ct is k_t = 2(m & 7) + ct, Re for
// m < 8 and Im otherwise (the kernel forms x(t) +- x(t + N_t/2)).
void t_forward_image(const Derived& dv, bool adjoint_of_inverse, float* dst) {
  const StreamCfg& sc = dv.sc;
  const dtst_desc& d = dv.d;
  const int ktp = 8 * sc.ct;
  const double ntot = double(d.n_global[0]) * d.n_global[1] * d.n_global[2] * d.n_global[3];
  const int tlim = sc.tf ? sc.nt / 2 : sc.nt;
  for (int h = 0; h < sc.th; ++h)
    for (int j = 0; j < 4; ++j)
      for (int ct = 0; ct < sc.ct; ++ct)
        for (int lane = 0; lane < 64; ++lane) {
          const int m = lane & 15, g = lane >> 4;
          const int t = 16 * h + 4 * g + j;
          const int c = 16 * ct + m;
          const bool is_re = sc.tf ? m < 8 : c < ktp;
          const int kt = sc.tf ? 2 * (m & 7) + ct : (is_re ? c : c - ktp);
          double v = 0.0;
          if (t < tlim && kt < sc.kt) {
            double re, im;
            bval(d, 3, kt, t, &re, &im);
            double s = adjoint_of_inverse ? half_weight(d.n_global[3], kt) / ntot : 1.0;
            v = s * (is_re ? re : im);
          }
          dst[((h * 4 + j) * sc.ct + ct) * 64 + lane] = static_cast<float>(v);
        }
}

// z image of the forward streaming kernel (A operand of the second MFMA,
// staged in LDS): float4 entry ((cl*ZT + zt)*MT + mt)*64 + lane, component
// i, holds row r = 16mt + m at z = 16zt + 4g + i of class cl; rows [0, KCP)
// are Re B_z[p][z], rows [KCP, 2KCP) are Im B_z[p][z], p = s*NCLS + cl.
// With MT = 1 (KCP = 8) row r holds slot s = 2(r >> 2) + ((r >> 1) & 1),
// Re for even r and Im for odd r, so that the products with Re B_z and Im B_z
// of one slot land in accumulator registers 2j and 2j + 1 of one lane.
// With t folded, the blocks hold the three-product operands of B = Br +
// i Bi: blocks mr < mt / 2 Br, the next mt / 2 blocks Bi - Br, the last
// mt / 2 Br + Bi, each for the rows (slots) of block mr.
void z_forward_image(const Derived& dv, float* dst) {
  const StreamCfg& sc = dv.sc;
  const dtst_desc& d = dv.d;
  const int nb = z_blocks(sc);
  for (int cl = 0; cl < sc.ncls; ++cl)
    for (int zt = 0; zt < sc.zt; ++zt)
      for (int mb = 0; mb < nb; ++mb)
        for (int lane = 0; lane < 64; ++lane)
          for (int i = 0; i < 4; ++i) {
            const int m = lane & 15, g = lane >> 4;
            const int z = 16 * zt + 4 * g + i;
            double v = 0.0;
            if (sc.tf) {
              const int half = sc.mt / 2, kind = mb / half, mr = mb % half;
              const int p = (16 * mr + m) * sc.ncls + cl;
              if (p < sc.kz && z < sc.zh) {
                double re, im;
                bval(d, 2, p, z, &re, &im);
                v = kind == 0 ? re : (kind == 1 ? im - re : re + im);
              }
            } else {
              const int row = 16 * mb + m;
              const bool is_re = sc.mt == 1 ? (row & 1) == 0 : row < sc.kcp;
              const int s = sc.mt == 1 ? 2 * (row >> 2) + ((row >> 1) & 1) : (is_re ? row : row - sc.kcp);
              const int p = s * sc.ncls + cl;
              if (p < sc.kz && z < sc.zh) {
                double re, im;
                bval(d, 2, p, z, &re, &im);
                v = is_re ? re : im;
              }
            }
            dst[((((size_t)cl * sc.zt + zt) * nb + mb) * 64 + lane) * 4 + i] = static_cast<float>(v);
          }
}

// t image of the inverse streaming kernel (A operand of its second MFMA):
// entry ((mt*CT + ct)*4 + i)*64 + lane holds A[t][c] with t = 16mt + m,
// c = 16ct + 4g + i: Re C_t[t][kt] for c < 8CT, -Im C_t[t][kt] otherwise,
// where C_t[t][kt] = scale(kt) conj(B_t[kt][t]).  t-folded (tf), only
// t < N_t/2 is filled and K index 4g + i of tile ct is
// k_t = 2(2g + (i & 1)) + (i >> 1), Re for ct = 0 and Im for ct = 1 (the
// rows of the three-product z expansion of the t-folded inverse).  With the
// four-class z fold of one column tile (MT = 1), K index 4g + i is
// k_t = 2g + (i & 1), Re for i < 2 and Im otherwise (Re and Im of one k_t in
// registers i and i + 2 of one lane of the z expansion).
void t_inverse_image(const Derived& dv, bool is_inverse, float* dst) {
  const StreamCfg& sc = dv.sc;
  const dtst_desc& d = dv.d;
  const int ktp = 8 * sc.ct;
  const double ntot = double(d.n_global[0]) * d.n_global[1] * d.n_global[2] * d.n_global[3];
  const int tlim = sc.tf ? sc.nt / 2 : sc.nt;
  for (int mt = 0; mt < sc.th; ++mt)
    for (int ct = 0; ct < sc.ct; ++ct)
      for (int i = 0; i < 4; ++i)
        for (int lane = 0; lane < 64; ++lane) {
          const int m = lane & 15, g = lane >> 4;
          const int t = 16 * mt + m;
          const int c = 16 * ct + 4 * g + i;
          // t-folded: tile ct holds part ct (0 Re, 1 -Im) of k_t = 2(2g + (i & 1)) + (i >> 1)
          const bool is_re = sc.tf ? ct == 0 : (sc.mt == 1 ? i < 2 : c < ktp);
          const int kt = sc.tf ? 2 * (2 * g + (i & 1)) + (i >> 1)
                               : (sc.mt == 1 ? 2 * g + (i & 1) : (is_re ? c : c - ktp));
          double v = 0.0;
          if (t < tlim && kt < sc.kt) {
            double re, im;
            bval(d, 3, kt, t, &re, &im);  // B_t = re + i im; conj(B_t) = re - i im
            const double s = is_inverse ? half_weight(d.n_global[3], kt) / ntot : 1.0;
            v = is_re ? s * re : s * im;  // -Im(s conj B_t) = s * im
          }
          dst[((mt * sc.ct + ct) * 4 + i) * 64 + lane] = static_cast<float>(v);
        }
}

// z image of the inverse streaming kernel (B operand of its first MFMA,
// staged in LDS): float4 entry ((cl*ZT + zt)*MT + q)*64 + lane, component
// i, holds row kz' = 16q + 4g + i at z = 16zt + m: Re C_z[z][p] for
// kz' < KCP and Im C_z[z][p] otherwise, C_z[z][p] = conj(B_z[p][z]).
// With MT = 1 (KCP = 8) row kz' holds slot s = 2g + (i >> 1), Re for even i
// and Im for odd i.
// With t folded, the blocks hold the three-product operands of C_z = Cr +
// i Ci (Cr = Re B, Ci = -Im B): blocks qh < mt / 2 Cr, the next mt / 2
// blocks Ci - Cr, the last mt / 2 Cr + Ci, each for the K entries of block qh.
void z_inverse_image(const Derived& dv, float* dst) {
  const StreamCfg& sc = dv.sc;
  const dtst_desc& d = dv.d;
  const int nb = z_blocks(sc);
  for (int cl = 0; cl < sc.ncls; ++cl)
    for (int zt = 0; zt < sc.zt; ++zt)
      for (int q = 0; q < nb; ++q)
        for (int lane = 0; lane < 64; ++lane)
          for (int i = 0; i < 4; ++i) {
            const int m = lane & 15, g = lane >> 4;
            const int z = 16 * zt + m;
            if (sc.tf) {
              const int half = sc.mt / 2, kind = q / half, qh = q % half;
              const int p = (16 * qh + 4 * g + i) * sc.ncls + cl;
              double v = 0.0;
              if (p < sc.kz && z < sc.zh) {
                double re, im;
                bval(d, 2, p, z, &re, &im);
                const double cr = re, ci = -im;
                v = kind == 0 ? cr : (kind == 1 ? ci - cr : cr + ci);
              }
              dst[((((size_t)cl * sc.zt + zt) * nb + q) * 64 + lane) * 4 + i] = static_cast<float>(v);
              continue;
            }
            const int kzp = 16 * q + 4 * g + i;
            const bool is_re = sc.mt == 1 ? (i & 1) == 0 : kzp < sc.kcp;
            const int s = sc.mt == 1 ? 2 * g + (i >> 1) : (is_re ? kzp : kzp - sc.kcp);
            const int p = s * sc.ncls + cl;
            double v = 0.0;
            if (p < sc.kz && z < sc.zh) {
              double re, im;
              bval(d, 2, p, z, &re, &im);
              v = is_re ? re : -im;
            }
            dst[((((size_t)cl * sc.zt + zt) * nb + q) * 64 + lane) * 4 + i] = static_cast<float>(v);
          }
}

// Axis image, float4 entries indexed by lane (m = lane & 15, g = lane >> 4)
// and component i.  With 3 parts (the axis kernels) part 0 holds Br, part 1
// Bi - Br, part 2 Br + Bi of the basis value Br + i Bi; with 2 parts (the y
// images of the fused stream kernels) part 0 Re, part 1 Im.  Entry layouts
// below with 2 parts; 3 parts stride the same way.
//   fold 0: entry ((kt*JQ + q)*2 + part)*64 + lane = basis[k][j],
//           k = 16kt + m, j = 16q + 4g + i.
//   fold 1: same entry layout; tile kt holds parity class c = (kt >= kth),
//           mode p = 2 (16 (kt - c kth) + m) + c, column j = 16q + 4g + i < J/2.
//   fold 2: entry (((kt*JQ + q)*2 + c)*2 + part)*64 + lane = basis[y][p],
//           y = 16kt + m < KO/2, mode p = 2 (16q + 4g + i) + c.
//   fold 3: fold 0's entry layout; tile kt holds class c = kt mod 4, mode
//           p = 4 (16 (kt / 4) + m) + c, column j = 16q + 4g + i < J/4.
//   fold 4: entry (((kt*JQ + q)*4 + c)*2 + part)*64 + lane = basis[y][p],
//           y = 16kt + m < KO/4, mode p = 4 (16q + 4g + i) + c.
// forward: basis[k][j] = B_dim[k][j]; inverse: basis[y][p] = conj(B_dim[p][y]).
void axis_image(const Derived& dv, const AxisCfg& a, int dim, bool inverse, float* dst) {
  const dtst_desc& d = dv.d;
  const int ncls = axis_image_classes(a);
  for (int kt = 0; kt < a.ktiles; ++kt)
    for (int q = 0; q < a.JQ; ++q)
      for (int c = 0; c < ncls; ++c)
        for (int part = 0; part < a.parts; ++part)
          for (int lane = 0; lane < 64; ++lane)
            for (int i = 0; i < 4; ++i) {
              const int m = lane & 15, g = lane >> 4;
              int k, j;  // output row, contracted index (before the basis orientation)
              bool ok;
              if (a.fold == 1) {
                const int cls = kt >= a.kth ? 1 : 0;
                k = 2 * (16 * (kt - cls * a.kth) + m) + cls;
                j = 16 * q + 4 * g + i;
                ok = k < a.KO && j < a.J / 2;
              } else if (a.fold == 2) {
                k = 16 * kt + m;
                j = 2 * (16 * q + 4 * g + i) + c;
                ok = k < a.KO / 2 && j < a.J;
              } else if (a.fold == 3) {
                k = 4 * (16 * (kt >> 2) + m) + (kt & 3);
                j = 16 * q + 4 * g + i;
                ok = k < a.KO && j < a.J / 4;
              } else if (a.fold == 4) {
                k = 16 * kt + m;
                j = 4 * (16 * q + 4 * g + i) + c;
                ok = k < a.KO / 4 && j < a.J;
              } else {
                k = 16 * kt + m;
                j = 16 * q + 4 * g + i;
                ok = k < a.KO && j < a.J;
              }
              double v = 0.0;
              if (ok) {
                double re, im;
                if (inverse) {
                  bval(d, dim, j, k, &re, &im);
                  im = -im;
                } else {
                  bval(d, dim, k, j, &re, &im);
                }
                if (a.parts == 3) v = part == 0 ? re : (part == 1 ? im - re : re + im);
                else v = part == 0 ? re : im;
              }
              dst[(((((size_t)kt * a.JQ + q) * ncls + c) * a.parts + part) * 64 + lane) * 4 + i] =
                  static_cast<float>(v);
            }
}

}  // namespace

void build_images(const Derived& dv, std::vector<float>* blob) {
  blob->assign(dv.img.total, 0.0f);
  float* b = blob->data();
  t_forward_image(dv, false, b + dv.img.t_fwd);
  t_forward_image(dv, true, b + dv.img.t_fwd_adjoint_of_inverse);
  z_forward_image(dv, b + dv.img.z_fwd);
  t_inverse_image(dv, true, b + dv.img.t_inv);
  t_inverse_image(dv, false, b + dv.img.t_inv_adjoint_of_forward);
  z_inverse_image(dv, b + dv.img.z_inv);
  axis_image(dv, dv.ay_f, 1, false, b + dv.img.y_fwd);
  axis_image(dv, dv.ax_f, 0, false, b + dv.img.x_fwd);
  axis_image(dv, dv.ay_i, 1, true, b + dv.img.y_inv);
  axis_image(dv, dv.ax_i, 0, true, b + dv.img.x_inv);
  if (dv.img.y_blk != dv.img.y_inv) axis_image(dv, dv.ay_b, 1, true, b + dv.img.y_blk);
  // the fused inverse + block epilogue's z and t images: those of the
  // inverse for its own z configuration
  Derived db = dv;
  db.sc = dv.sb;
  z_inverse_image(db, b + dv.img.z_blk);
  t_inverse_image(db, true, b + dv.img.t_blk);
}

void plain_basis(const dtst_desc& d, int dim, int kind, float* out) {
  const int64_t K = dim < 3 ? 2 * int64_t(d.kmax[dim]) : d.kt;
  const int64_t n = d.n_local[dim];
  for (int64_t p = 0; p < K; ++p)
    for (int64_t j = 0; j < n; ++j) {
      double re, im;
      bval(d, dim, p, j, &re, &im);
      out[(p * n + j) * 2 + 0] = static_cast<float>(re);
      out[(p * n + j) * 2 + 1] = static_cast<float>(kind == 1 ? -im : im);
    }
}

}  // namespace dtst
