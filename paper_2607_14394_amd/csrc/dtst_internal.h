// Internal declarations shared by the host tables, the C ABI and the HIP
// kernels of the DTST library.  Not part of the public interface.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "dtst.h"

namespace dtst {

// ---------------------------------------------------------------------------
// Streaming t+z kernels (forward: real rows -> (Kz x Kt) complex rows;
// inverse: the mirror).  One "row" is the contiguous (N_z x N_t) block of a
// fixed (b, c, x, y).
//
//   CT   number of 16-wide column tiles holding (Re kt | Im kt): 1 if kt <= 8
//        (columns 0..7 = Re, 8..15 = Im), 2 if kt <= 16 (tile 0 Re, tile 1 Im)
//   TH   number of 16-wide t groups: N_t padded to 16*TH, t = 16h + 4g + j
//   MT   16-row tiles per z class: rows [0, KCP) = Re, [KCP, 2 KCP) = Im,
//        KCP = 8*MT slots per class
//   NCLS 1, or 2 when z is folded: with N_z^loc = N_z even,
//        B[k, z + N/2] = (-1)^k B[k, z], so even k see x[z] + x[z+N/2] and
//        odd k see x[z] - x[z+N/2]; class c holds the modes p = 2s + c.
//        4 when in addition N_z % 4 == 0, k_max(z) is even, CT = 2 and
//        K_z <= 64 (MT = 2):
//        B[k, z + N/4] = (-i)^k B[k, z], classes by k mod 4 (p = 4s + c),
//        each contracting the z < N/4 combination sum_j (-i)^(cj) x[z + jN/4].
// ---------------------------------------------------------------------------
struct StreamCfg {
  int ct = 1, th = 1, mt = 2, ncls = 1;
  int nt = 0, nz = 0, kt = 0, kz = 0;
  int zh = 0;   // z extent per class pass (N_z / ncls)
  int zt = 0;   // ceil(zh / 16)
  int kcp = 0;  // padded slots per class = 8*mt
  int vec = 0;  // 1 when N_t % 4 == 0 (16-byte row chunks)
  // 1 when t folds: CT = 2, N_t = 32 and the shard holds the whole t extent
  // (the t images then hold the folded layout of the split kernels)
  int tf = 0;
  size_t lds_bytes = 0;
  // Fused t + z + y (fwd_tzy_kernel) and y + z + t (inv_yzt_kernel), used
  // when fuse_y is set:
  //   ncy        y classes: 2 when y is folded (slot = row pair), else 1
  //   kyt        16-wide tiles of K_y per class: k tiles of the forward y
  //              image, K steps of the inverse y image
  //   fused_mrow LDS row stride (complex values) of the exchanged row results
  //   fused_y_lds 1 when the y basis images are staged in LDS (else read from
  //              global memory)
  int fuse_y = 0, ncy = 1, kyt = 1, fused_mrow = 0, fused_y_lds = 0;
  size_t fused_lds_bytes = 0;
  // filled at plan creation on the plan's device (prepare_stream)
  int grid_fwd = 0, grid_inv = 0;  // resident workgroups of each kernel
  int grid_fused = 0;  // resident workgroups of fwd_tzy_kernel
};

// Generic complex contraction along a middle axis:
//   out[b][k][n] (+)= sum_j basis[k][j] in[b][j][n],
// b < nb, j < J, k < KO, n < NN (complex elements).
//
// fold 1 (forward, the contracted spatial axis is the whole even extent):
//   the K loop runs over j < J/2 with in[j] +- in[j + J/2]; k tiles
//   [0, kth) hold the even modes p = 2s, tiles [kth, 2 kth) the odd ones.
// fold 2 (inverse, the output spatial axis is the whole even extent): the K
//   loop runs over the J/2 even and J/2 odd modes; k tiles cover rows
//   y < KO/2 and write E + O at y and E - O at y + KO/2.
struct AxisCfg {
  int64_t nb = 0;
  int J = 0, KO = 0, NN = 0;
  int fold = 0;
  int JQ = 0;      // 16-wide K steps
  int ktiles = 0;  // 16-row k tiles
  int kth = 0;     // fold 1: k tiles per parity class
  // parts per image entry: 3 for the axis kernels (Br, Bi - Br, Br + Bi, the
  // factors of their three-product form), 2 (Re, Im) for the y images of the
  // fused stream kernels
  int parts = 3;
};

// Float offsets of each kernel-ready image inside the plan's device blob.
struct Images {
  size_t t_fwd = 0, t_fwd_adjoint_of_inverse = 0;  // streaming forward, B operand
  size_t z_fwd = 0;                                // streaming forward, LDS image
  size_t t_inv = 0, t_inv_adjoint_of_forward = 0;  // streaming inverse, A operand
  size_t z_inv = 0;                                // streaming inverse, LDS image
  size_t y_fwd = 0, x_fwd = 0, y_inv = 0, x_inv = 0;  // axis images
  size_t z_blk = 0, t_blk = 0;                         // fused inverse + block epilogue
  size_t y_blk = 0;  // y expansion of dtst_inverse_block (y_inv unless the plan fuses y)
  size_t total = 0;
};

struct Derived {
  dtst_desc d{};
  int64_t K[4] = {0, 0, 0, 0};
  int64_t M = 0;
  StreamCfg sc;
  AxisCfg ay_f, ax_f, ax_i, ay_i;  // per-channel shapes; nb is per (b, c) below
  AxisCfg ay_b;                    // the inverse y of dtst_inverse_block's separate y launch
  size_t ws_bytes = 0;
  size_t w1_bytes = 0;  // workspace offset of W2 (0 with the fused y: no W1)
  Images img;
  // Fused inverse + block epilogue (inv_zt_block_kernel): its z + t
  // configuration (z folded into at most 2 classes), whether dtst_inverse_block
  // uses it, the workspace it needs (W1 then W2), and its resident grid (set
  // at plan creation on the plan's device).
  StreamCfg sb;
  int blk = 0;
  size_t blk_ws_bytes = 0, blk_w1_bytes = 0;
  int grid_blk = 0;
};

// Host-side validation and derivation (pure C++; no HIP).
dtst_status derive(const dtst_desc* d, uint32_t flags, Derived* out, std::string* err);
// Build every image of the blob (fp64 maths, rounded to fp32 once).
void build_images(const Derived& dv, std::vector<float>* blob);
// Plain (K x N_loc) complex fp32 basis of one dimension (kind 0: B, 1: conj B).
void plain_basis(const dtst_desc& d, int dim, int kind, float* out);

// Retained stored index of position p along dimension dim (0..3).
int64_t retained_index(const dtst_desc& d, int dim, int64_t p);

// ---------------------------------------------------------------------------
// Kernel launchers (defined in the .hip sources).  All return hipSuccess or
// the launch error as an int (hipError_t).
// ---------------------------------------------------------------------------
// Sets kernel attributes and resident-grid sizes for the current device.
int prepare_stream(StreamCfg* c);
int launch_fwd_tz(const StreamCfg& c, const float* x, void* out, int64_t rows,
                  const float* timg, const float* zimg, void* stream);
// Forward t + z + y of `planes` (b, c, x) planes of ny rows into the
// (planes x K_y x K_z K_t) complex output; ay is the forward y contraction
// whose image (yimg) supplies the y basis.
int launch_fwd_tzy(const StreamCfg& c, const AxisCfg& ay, const float* x, void* out, int64_t planes, int ny,
                   const float* timg, const float* zimg, const float* yimg, void* stream);
// Inverse y + z + t of `planes` planes: (planes x K_y x K_z K_t) complex in,
// (planes x ny x N_z x N_t) real out; ay is the inverse y expansion whose
// image (yimg) supplies the y basis.
int launch_inv_yzt(const StreamCfg& c, const AxisCfg& ay, const void* in, float* y, int64_t planes, int ny,
                   const float* timg, const float* zimg, const float* yimg, void* stream);
int launch_inv_zt(const StreamCfg& c, const void* in, float* y, int64_t rows,
                  const float* timg, const float* zimg, void* stream);
// Fused inverse z + t expansion and block epilogue (k_block_zt.hip):
//   y[b,o,.] = GELU(w x[b,.,.] + zt-expansion of in[b,o,.]) over the
// batch * nxy (b, x, y) rows; in is the y-expanded spectrum
// (B, C_out, N_x, N_y, K_z, K_t), c its z + t configuration (Derived::sb).
size_t block_zt_lds_bytes(const StreamCfg& c, int64_t ci, int64_t co);
bool block_zt_supported(const StreamCfg& c, int64_t ci, int64_t co);
int prepare_block_zt(const StreamCfg& c, int64_t ci, int64_t co, int* grid);
int launch_inv_zt_block(const StreamCfg& c, int grid_resident, const void* in, const float* x, const float* w,
                        float* y, int64_t batch, int64_t nxy, int64_t ci, int64_t co, const float* timg,
                        const float* zimg, void* stream);
int launch_axis(const AxisCfg& c, int64_t nb, const void* in, void* out, const float* img,
                int accumulate, void* stream);
// LDS bytes of one workgroup of the mix kernels (mix, mix_h and wgrad alike).
size_t mix_lds_bytes(int64_t B, int64_t ci, int64_t co);
// Largest C_out the mix kernels cover (64 lanes x 8 columns per row).
constexpr int64_t kMixMaxCout = 512;
int launch_mix(const void* xhat, const void* w, void* yhat, int64_t B, int64_t ci, int64_t co,
               int64_t M, int64_t m0, int64_t m1, void* stream);
int launch_mix_h(const void* gy, const void* w, void* gx, int64_t B, int64_t ci, int64_t co,
                 int64_t M, int64_t m0, int64_t m1, void* stream);
// y <- GELU(w x + y) over B batch entries of V points (block epilogue).
int launch_block_epilogue(const float* x, const float* w, float* y, int64_t B, int64_t ci, int64_t co, int64_t V,
                          void* stream);
// y = act(w x + bias) over B batch entries of V points (lift / projection);
// bias may be null (zero); act 1 = GELU.
int launch_pointwise(const float* x, const float* w, const float* bias, float* y, int64_t B, int64_t ci, int64_t co,
                     int64_t V, int act, void* stream);
int launch_wgrad(const void* xhat, const void* gy, void* gw, int64_t B, int64_t ci, int64_t co,
                 int64_t M, int64_t m0, int64_t m1, int accumulate, void* stream);

// Bytes of the per-device scratch array that dtst_forward_noalloc uses as its
// workspace (k_scratch.hip).
constexpr size_t kScratchBytes = DTST_SCRATCH_BYTES;
// Device address of `device`'s scratch array, looked up with that device
// current on the first call and kept; hipSuccess or the HIP error.
int scratch_address(int device, void** out);

}  // namespace dtst
