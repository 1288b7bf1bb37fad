// Argument blocks and launchers of the memory-bound PI-GAN kernels.
#pragma once
#include "common.h"

namespace pigan {

template <class T> struct FirstArgs {
  const float* p1; int64_t p_g; int in_dim; int d; int W;  // fp32 master W1 (row-major [W][in_dim])
  const float* zp; int64_t zp_g;                           // per-sample z-projection + b1
  const float* x; int64_t x_g; int x_shared; int64_t Pn;   // locations; Pn points per sample
  T* out_a; T* out_h; int64_t o_g; int64_t ldo;
  Seg seg;
  int exact;                                               // fp32 storage: tanh in fp64
};

struct ResidArgs {
  const float* jY; int64_t jy_g; int64_t offY;   // Y jets: value at offY, d/dx_i at offY + (1+i)*plane
  const float* jU; int64_t ju_g; int64_t offU;   // u jets: d/dx_i at offU+(1+i)*plane, d2 at offU+(1+d+i)*plane
  int64_t plane; int64_t M; int d;
  const float* f; int64_t f_g; float f_const;
  float* r; int64_t r_g;
  float* gY; float* gU;                          // cotangent vectors (same layout as the jets) or null
  const float* gq; int64_t gq_g;                 // extra cotangent of r per point (critics of the free sensors) or null
  const float* w_group; float qscale;            // q = qscale * w_g * r
  double* part;                                  // [G][blocks] partial sums of r^2, or null
};

template <class T> struct OutBwdArgs {
  const T* A; T* dA; int64_t o_g; int64_t ldo;   // saved pre-activation of the top layer, its cotangent
  const float* gbar; int64_t gb_g;               // output cotangents (jet layout)
  const float* wout; int64_t w_g;                // w_out (W) followed by b_out
  int W; int64_t ppb;                            // points per block
  double* part; int n_slots; int slot0;          // [G][n_slots][W+1] fp64 partials
  Seg seg;
  int exact;                                     // fp32 storage: tanh in fp64
};

// output layer of a shared trunk (two heads), reverse pass
template <class T> struct Out2BwdArgs {
  const T* A; const T* H; T* dA; T* gh; int64_t o_g; int64_t ldo;  // top pre-activation / activation; outputs
  const float* gbar0; const float* gbar1; int64_t gb_g;        // cotangents of the Y and u heads (jet layout)
  const float* wout; int64_t w_g;                              // [w_Y (W), b_Y, w_u (W), b_u]
  int W; int64_t ppb;                                          // points per block
  double* part; int n_slots; int slot0;                        // [G][n_slots][2 (W+1)] fp64 partials
  Seg seg;
  int exact;                                                   // fp32 storage: tanh in fp64
};

template <class T> struct FirstBwdArgs {
  const float* dAs; int64_t as_g; int64_t ldas;  // sensor rows (fp32) [n_sen][W]
  const T* dA; int64_t a_g; int64_t lda;         // collocation stream rows: stream k at k * n_col
  int64_t n_sen; int64_t n_col;
  int n_s; int P; int S; int W; int d; int nd1;
  const float* xs; int64_t xs_g;                 // sensor locations [n_s][d]
  const float* xc; int64_t xc_g;                 // collocation points of the chunk [S][P][d]
  int nrc;                                       // row chunks per sample (blocks per sample)
  double* part;                                  // [G][S][nrc][7][W]
};

hipError_t launch_zproj(const float* p1, int64_t p_g, int in_dim, int d, int W, const float* z, int64_t z_g,
                        int n_z, int S, float* zp, int64_t zp_g, int G, hipStream_t st);
template <class T> hipError_t launch_first_fwd(int nd1, int nd2, const FirstArgs<T>& a, int G, hipStream_t st);
template <class T>
hipError_t launch_out_fwd(const T* H, int64_t h_g, int64_t ldh, int64_t R, int64_t n_value, int W,
                          const float* wout, int64_t w_g, float* y, int64_t y_g, int G, hipStream_t st);
hipError_t launch_residual(const ResidArgs& a, int G, hipStream_t st);
int residual_blocks(int64_t M);
hipError_t launch_sum_partials(const double* part, int nb, double* acc, int acc_stride, int slot, int G,
                               hipStream_t st);
template <class T>
hipError_t launch_snap_fill(const float* yY, int64_t yY_g, const float* yU, int64_t yU_g, int nY, int nU,
                            int n_fake, const float* real, int64_t real_g, int n_real, int n_in, T* X,
                            int64_t x_g, int ldx, int G, hipStream_t st);
hipError_t launch_disc_seed(const float* score, int64_t sc_g, int n_fake, int n_real, int S_total, int B_total,
                            const float* w_group, float loss_scale, float* seed, double* acc, int acc_stride,
                            int G, hipStream_t st);
int out_bwd_blocks(int64_t n_points, int ppb);
template <class T>
// fake row i: Y values yY[i * ldY + j], u values yU[i * ldU + offU + j]
hipError_t launch_gp_mix(const float* yY, int64_t yY_g, const float* yU, int64_t yU_g, int nY, int nU, int ldY,
                         int ldU, int offU, const float* real, int64_t real_g, const float* eps, int64_t eps_g, int b0,
                         int n, int n_in, T* X, int64_t x_g, int ldx, int G, hipStream_t st);
hipError_t launch_fill2(float* seed, int64_t s_g, int n, float v0, float v1, int two, int G, hipStream_t st);
template <class T>
hipError_t launch_gp_norm(const float* gin, int64_t g_g, int n, int n_in, const float* w_group, float scale,
                          double* part, int64_t p_g, T* X, int64_t x_g, int ldx, int G, hipStream_t st);
template <class T> hipError_t launch_out_bwd(int nd1, int nd2, const OutBwdArgs<T>& a, int G, hipStream_t st);
template <class T> hipError_t launch_out2_bwd(int nd1, int nd2, const Out2BwdArgs<T>& a, int G, hipStream_t st);
// snapshot rows from sensor values laid out ld apart per sample (u values
// offU into the row), then the real rows
template <class T>
hipError_t launch_snap_fill_rows(const float* yY, int64_t yY_g, const float* yU, int64_t yU_g, int nY, int nU,
                                 int ld, int offU, int n_fake, const float* real, int64_t real_g, int n_real, int n_in,
                                 T* X, int64_t x_g, int ldx, int G, hipStream_t st);
hipError_t launch_concat_rows(const float* a, int64_t a_g, int na, const float* b, int64_t b_g, int nb, int d,
                              float* out, int64_t o_g, int G, hipStream_t st);
hipError_t launch_fill_f32(float* p, int64_t n, int64_t p_g, float v, int G, hipStream_t st);

// domain decomposition: the snapshots of D critics (one per subdomain) and the
// scatter of their input cotangents back to the generator's outputs
struct HierSnap {
  const float* jY; const float* jU; int nsY; int nsU;    // sensor values of the chunk:
  int ldY; int ldU; int offU;                            //   jY[s * ldY + i], jU[s * ldU + offU + i]
  const float* r; const float* f; float f_const;         // residual [s * P + p]; source (chunk view) or null
  const float* xc; int P; int d;                         // collocation points of the chunk [s][P][d]
  const int32_t* idxY; const int32_t* idxU; const int32_t* idxF;  // [D][mY], [D][mU], [D][nF]
  int mY; int mU; int nF; int n_in;
  int32_t* bad;                                          // set to 1 on an index out of range
};
template <class T>
hipError_t launch_hier_snap(const HierSnap& h, int n_fake, const float* real, int64_t real_g, int n_real, T* X,
                            int64_t x_g, int ldx, int D, hipStream_t st, const float* eps = nullptr,
                            int64_t eps_g = 0, int b0 = 0);
hipError_t launch_hier_scatter(const HierSnap& h, const float* dX, int64_t dx_g, int ldx, int n_fake, int D,
                               float* gY, float* gU, float* gN, hipStream_t st);
// loss[k][2] = lambda_pde * acc[slot] / SP for every critic k
hipError_t launch_hier_pde_loss(const double* acc, int slot, float lambda_pde, int64_t SP, float* loss, int D,
                                int32_t* nonfinite, hipStream_t st);
// dst[(col/Jp)*J + col%Jp] (+)= scale * sum_slots part[g][slot][col]  (fp64, fixed order)
template <class Tin>
hipError_t launch_colsum(const Tin* part, int64_t p_g, int n_slots, int64_t slot_stride, int64_t ncols, int Jp, int J,
                         float* dst, int64_t d_g, int accumulate, float scale, int32_t* nonfinite, int G,
                         hipStream_t st);
template <class T> hipError_t launch_first_bwd(const FirstBwdArgs<T>& a, int G, hipStream_t st);
hipError_t launch_first_wgrad(const double* part, int S, int nrc, int W, int d, int nd1, int in_dim, const float* z,
                              int64_t z_g, int n_z, float* grad, int64_t g_g, int accumulate, float scale,
                              int32_t* nonfinite, int G, hipStream_t st);
hipError_t launch_losses(const double* acc, int acc_stride, const float* w_group, int S, int B, int64_t SP,
                         float lambda_pde, float lambda_gp, int n_gp, float* loss, float* gp, int32_t* nonfinite,
                         int G, hipStream_t st);
hipError_t launch_zero(double* acc, int n, int32_t* flag, hipStream_t st);
template <class T>
hipError_t launch_cast(const float* src, int64_t s_g, int N, int K, int Kp, T* dst, T* dstT, int64_t d_g, int G,
                       hipStream_t st);
// split-product weight copies (pair-blocked bf16 pieces in fp32-pitch rows)
hipError_t launch_cast_pair(const float* src, int64_t s_g, int N, int K, int Kp, float* dst, float* dstT, int64_t d_g,
                            int G, hipStream_t st);
// two-term weights [hi | lo] per row (16-bit storage), rows 2 K wide
template <class T>
hipError_t launch_cast2(const float* src, int64_t s_g, int N, int K, T* dst, int64_t d_g, int G, hipStream_t st);

}  // namespace pigan
