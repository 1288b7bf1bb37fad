/*
 * pigan.h — C ABI of the MI355X PI-GAN training-step library (libpigan.so).
 *
 * The library evaluates the physics-informed GAN of arXiv 1910.13444 on one
 * AMD MI355X (gfx950): tanh-MLP generators for the log-conductivity Y = log k
 * and the hydraulic head u, both taking one location x plus the noise vector z
 * as a narrow input (Sec. III.C, "Single Node optimizations"); first and second
 * spatial derivatives carried through every layer so that the Darcy residual
 * -div(exp(Y) grad u) - f can be formed (Eq. 1 with k = exp(Y), Eq. 2;
 * the paper induces this f-network by automatic differentiation,
 * Sec. III.B.1); a tanh-MLP discriminator on whole sensor snapshots
 * (Sec. III.C); WGAN critic losses weighted per subdomain (Sec. III.B.1);
 * and fp32 gradients of every weight with half-precision activations
 * (Sec. III.C, mixed precision).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every pointer argument is a DEVICE pointer owned by the caller unless
 *    stated otherwise.  The library never allocates device memory, never frees
 *    caller memory and keeps no state between calls besides a thread-local
 *    error string (and, when enabled, the profiling record).  The one
 *    exception is pigan_train_step_grads_noalloc, which works in a fixed
 *    device array of the library instead of a caller workspace.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Calls enqueue work
 *    on it and return; outputs are valid after the caller synchronises it.
 *  - Argument checks run on the host before anything is enqueued; a non-OK
 *    status means nothing was launched (except PIGAN_EDEVICE, which reports a
 *    HIP launch/runtime error).  pigan_last_error() describes the failure.
 *  - MLP parameters are fp32, packed per group as
 *      [W1 (width x in_dim, row-major), b1, W2 (width x width), b2, ...,
 *       W_L, b_L, w_out (width), b_out]
 *    and groups are stacked contiguously: params[g * n_params + i].
 *  - Generator input order is [x_1..x_d, z_1..z_nz] (in_dim = d + n_z).
 *  - The arithmetic type (pigan_dtype) selects the storage and matrix-core
 *    operand type of the generators' hidden layers at the collocation points
 *    (the residual's jets); in bf16/fp16 their forward products take the
 *    fp32 weights as two terms, hi + lo in that type.  The adversarial path --
 *    the generators at the sensors and the discriminator -- is stored in fp32
 *    in every mode, with products from two bf16 pieces per fp32 operand in
 *    bf16/fp16 modes and from the fp64 matrix core in fp32 mode (there tanh
 *    and its derivatives are evaluated in fp64).  At the initial weights the
 *    critic responds far less to a uniform shift of a sensor block than to
 *    single sensors, so the sensor-row gradients are small differences of
 *    large terms and need the extra precision.  Accumulation, the first
 *    generator layer, the residual, losses and gradients are fp32 or wider.
 *  - Results are deterministic run to run (fixed-order reductions, no float
 *    atomics).
 */
#ifndef PIGAN_H
#define PIGAN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PIGAN_OK = 0,
  PIGAN_EINVAL = 1,      /* null pointer, non-positive size, inconsistent shapes */
  PIGAN_ENOTSUP = 2,     /* valid request the library does not implement */
  PIGAN_EWORKSPACE = 3,  /* workspace missing or smaller than required */
  PIGAN_EDEVICE = 4      /* HIP launch or runtime error */
} pigan_status;

typedef enum {
  PIGAN_FP32 = 0,        /* fp32 storage, fp32 matrix cores (fp64 on the adversarial path) */
  PIGAN_BF16 = 1,        /* bf16 storage (round-to-nearest-even), fp32 accumulate */
  PIGAN_FP16 = 2         /* fp16 storage (round-to-nearest-even), fp32 accumulate */
} pigan_dtype;
/* Descriptor fields and arguments that carry a pigan_dtype are int32_t, so
 * that any value a caller passes is well defined and rejected (EINVAL) when it
 * is none of the above. */

/* Shape of one tanh MLP: n_hidden tanh layers of `width` units on `in_dim`
 * inputs, then a linear scalar output.  `n_groups` independent copies
 * (subdomains) share the shape.  width must be a multiple of 32 and at most
 * 4096; n_hidden >= 1; in_dim >= 1. */
typedef struct {
  int32_t n_groups;
  int32_t in_dim;
  int32_t n_hidden;
  int32_t width;
} pigan_mlp;

/* Number of fp32 parameters of one group of `net` (see packing above). */
int64_t pigan_mlp_n_params(const pigan_mlp* net);

/*
 * pigan_gen_forward — generator values and spatial jets (Sec. III.B.1: the
 * generator represents log k and u from a location and a noise vector; the
 * differential operator is applied to it analytically).
 *
 *   net    : generator shape; net->in_dim must equal d + n_z.
 *   params : [G, n_params] fp32.
 *   d      : spatial dimensions, 1..3.
 *   z      : [G, S, n_z] fp32 noise vectors.
 *   x      : [G, S, P, d] fp32 locations, or [G, P, d] when x_shared != 0
 *            (the same P locations for every sample).
 *   order  : 0 value only; 1 adds d/dx_i; 2 adds d^2/dx_i^2 (no mixed terms).
 *   jet    : [G, 1 + order*d, S, P] fp32 output, components in the order
 *            value, d/dx_1..d/dx_d, d^2/dx_1^2..d^2/dx_d^2.
 *   ws     : device workspace of at least pigan_gen_forward_workspace() bytes,
 *            256-byte aligned.
 */
size_t pigan_gen_forward_workspace(const pigan_mlp* net, int32_t d, int32_t S, int32_t P,
                                   int32_t order, int32_t dt);
pigan_status pigan_gen_forward(const pigan_mlp* net, const float* params, int32_t d,
                               const float* z, const float* x, int32_t x_shared,
                               int32_t S, int32_t P, int32_t order, int32_t dt,
                               float* jet, void* ws, size_t ws_bytes, void* stream);

/*
 * pigan_pde_residual — Darcy residual r = -div(exp(Y) grad u) - f
 * = -exp(Y) (sum_i dY/dx_i du/dx_i + sum_i d^2u/dx_i^2) - f  (Eq. 1, Eq. 2).
 * The sign convention puts the operator on the left with a minus sign, so
 * f here is the negative of the paper's right-hand side (the paper's data use
 * f = 0).
 *
 *   jetY : [G, 1 + d, M] fp32 (value, d/dx_i) — layout of pigan_gen_forward
 *          with order 1 and M = S*P.
 *   jetU : [G, 1 + 2d, M] fp32 (value unused, d/dx_i, d^2/dx_i^2).
 *   f    : [G, M] fp32, or NULL to use the constant f_const everywhere.
 *   r    : [G, M] fp32 output.
 */
pigan_status pigan_pde_residual(int32_t d, int32_t G, int64_t M, const float* jetY,
                                const float* jetU, const float* f, float f_const, float* r,
                                void* stream);

/*
 * pigan_disc_forward — discriminator scores D(v) = w_out . h_L + b_out,
 * h_l = tanh(W_l h_{l-1} + b_l), h_0 = v, one whole snapshot per row
 * (Sec. III.C: the discriminator receives all sensors of its subdomain as a
 * single input).
 *
 *   snap  : [G, B, in_dim] fp32 snapshots.
 *   score : [G, B] fp32 output.
 */
size_t pigan_disc_forward_workspace(const pigan_mlp* net, int32_t B, int32_t dt);
pigan_status pigan_disc_forward(const pigan_mlp* net, const float* params, const float* snap,
                                int32_t B, int32_t dt, float* score, void* ws,
                                size_t ws_bytes, void* stream);

/*
 * One training step of the PI-GAN (Sec. III.B.1 and Sec. III.C).
 *
 * Per group g with weight w_g (the paper weights a subdomain's critic by
 * 1/(levels * subdomains in its level)):
 *   fake snapshot F_s = [Y(xsY_j, z_s)]_j || [u(xsU_j, z_s)]_j,  s < S
 *   r_{s,p}         = -exp(Y)(grad Y . grad u + lap u) - f  at (xc_{s,p}, z_s)
 *   L_D   = w_g (mean_s D(F_s) - mean_b D(real_b))
 *   L_adv = -w_g mean_s D(F_s)
 *   L_pde = w_g lambda_pde mean_{s,p} r^2
 * Outputs: gD = dL_D/d(disc params), gY = d(L_adv + L_pde)/d(Y params),
 * gU = d(L_adv + L_pde)/d(u params).  Gradients are OVERWRITTEN (not
 * accumulated).  The step is exactly additive over noise samples, so the
 * library processes samples in chunks of chunk_S (0 = the largest chunk whose
 * workspace stays within 128 GiB); the result does not depend on the chunking
 * up to fp32 summation order.
 */
typedef struct {
  pigan_mlp genY, genU, disc;  /* equal n_groups; genY/genU in_dim = d + n_z;
                                  disc in_dim = n_sY + n_sU */
  int32_t d, n_z;              /* d in 1..3 */
  int32_t S, P;                /* noise samples, collocation points per sample */
  int32_t n_sY, n_sU;          /* Y and u sensors per group (>= 1 each) */
  int32_t B_r;                 /* real snapshots per group */
  int32_t chunk_S;             /* samples per chunk, 0 = automatic */
  int32_t dt;                  /* a pigan_dtype value */
  float lambda_pde;            /* weight of the residual penalty (>= 0) */
  float lambda_gp;             /* critic gradient-penalty weight (>= 0); must be 0 for
                                  pigan_train_step_grads (ENOTSUP otherwise), any value for
                                  pigan_train_step_grads_gp */
  float loss_scale;            /* static loss scale (> 0; 1 unless fp16) */
  int32_t critic_only;         /* 0: every gradient; 1: the critic's update only -- gD, L_D
                                  and L_adv as in the full step; the generators run at the
                                  sensors only (no collocation rows, no residual: L_pde is
                                  reported as 0) and have no reverse pass; their gradient
                                  outputs are neither written nor required (may be NULL) */
} pigan_step_desc;

size_t pigan_workspace_bytes(const pigan_step_desc* s);

/*
 *   pY, pU, pD : [G, n_params] fp32 master weights.
 *   z   : [G, S, n_z]; xc : [G, S, P, d] collocation points (per sample);
 *   xsY : [G, n_sY, d], xsU : [G, n_sU, d] sensor locations (shared by all
 *         samples); f : [G, S, P] or NULL (then f_const);
 *   real: [G, B_r, n_sY + n_sU] real snapshots; w_group : [G] or NULL (= 1).
 *   gY, gU, gD : [G, n_params] fp32 outputs.
 *   loss : [G, 3] fp32 output (L_D, L_adv, L_pde).
 *   nonfinite : one device int32, set to 1 when any gradient or loss is not
 *               finite (the caller's loss-scaling logic skips such a step),
 *               else 0.
 */
pigan_status pigan_train_step_grads(const pigan_step_desc* s, const float* pY, const float* pU,
                                    const float* pD, const float* z, const float* xc,
                                    const float* xsY, const float* xsU, const float* f,
                                    float f_const, const float* real, const float* w_group,
                                    float* gY, float* gU, float* gD, float* loss,
                                    int32_t* nonfinite, void* ws, size_t ws_bytes, void* stream);

/*
 * pigan_train_step_grads_noalloc — for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same step, the same kernels and the same results as
 * pigan_train_step_grads, with its workspace in a fixed array of the library
 * (PIGAN_NOALLOC_SCRATCH_BYTES per device, held from the first call on a
 * device until the process ends) instead of a caller buffer.  It allocates
 * nothing itself.
 *   Returns PIGAN_EWORKSPACE, and launches nothing, when the step needs more
 *   than PIGAN_NOALLOC_SCRATCH_BYTES (pigan_workspace_bytes of the same
 *   descriptor; a smaller chunk_S lowers it).  lambda_gp must be 0.
 *   Every call on one device shares that device's array: calls whose work
 *   overlaps on a device (other streams, other host threads) race; serialise
 *   them.  The step initialises every workspace byte it reads, so no clearing
 *   is needed between calls.
 */
#define PIGAN_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
pigan_status pigan_train_step_grads_noalloc(const pigan_step_desc* s, const float* pY, const float* pU,
                                            const float* pD, const float* z, const float* xc,
                                            const float* xsY, const float* xsU, const float* f,
                                            float f_const, const float* real, const float* w_group,
                                            float* gY, float* gU, float* gD, float* loss,
                                            int32_t* nonfinite, void* stream);

/*
 * pigan_train_step_grads plus the critic's gradient penalty, the member of the
 * WGAN family the paper cites for its critics (Sec. I.C, Sec. II.C):
 *   x_b = eps_b real_b + (1 - eps_b) F_b,   b < n_gp = min(S, B_r)
 *         (fake snapshot b is noise sample b),
 *   P_g = w_g lambda_gp mean_b (||grad_v D(x_b)||_2 - 1)^2.
 * P_g is added to L_D (loss[g][0]) and its gradient to gD; gY and gU are
 * unchanged.  The weight gradient is the reverse pass of the critic's
 * directional derivative along c_b = dP/d(grad_v D(x_b)) (a pair whose input
 * gradient is exactly zero contributes to P but not to the gradient).
 *   gp_eps : [G, n_gp] fp32 mixing weights (device), required when
 *            lambda_gp > 0 (EINVAL if NULL); unused when lambda_gp = 0.
 *   gp     : [G] fp32 output P_g (device) or NULL.
 * Everything else as pigan_train_step_grads; pigan_workspace_bytes accounts
 * for the penalty's buffers when lambda_gp > 0.
 */
pigan_status pigan_train_step_grads_gp(const pigan_step_desc* s, const float* pY, const float* pU,
                                       const float* pD, const float* z, const float* xc,
                                       const float* xsY, const float* xsU, const float* f,
                                       float f_const, const float* real, const float* w_group,
                                       const float* gp_eps, float* gY, float* gU, float* gD,
                                       float* loss, float* gp, int32_t* nonfinite, void* ws,
                                       size_t ws_bytes, void* stream);

/*
 * Shared-trunk generator: the paper's own generator (Sec. III.C, "Single Node
 * optimizations"), one set of weights producing both log k and u.  A tanh
 * trunk on [x ; z] of L layers of width W (the paper uses 5 x 128, 11 x 512
 * and 21 x 1024); after the first layer every pair of layers is a residual
 * block, h_l = tanh(W_l h_{l-1} + b_l) + h_{l-2} for odd l >= 3 (skips for
 * gradient propagation, same section), then a linear head with two outputs,
 * Y = w_Y . h_L + b_Y and u = w_u . h_L + b_u.  The spatial jets of the trunk
 * carry 1 + 2d streams at the collocation points (u needs d2/dx_i2; Y uses
 * the value and first-derivative streams of the same trunk).
 *
 * Packing per group (fp32): [W1 (W x in_dim), b1, W2, b2, ..., W_L, b_L,
 *                            w_Y (W), b_Y, w_u (W), b_u].
 */
int64_t pigan_trunk_param_count(const pigan_mlp* trunk);

typedef struct {
  pigan_mlp trunk, disc;       /* equal n_groups; trunk in_dim = d + n_z;
                                  disc in_dim = n_sY + n_sU */
  int32_t d, n_z, S, P;        /* as pigan_step_desc */
  int32_t n_sY, n_sU, B_r, chunk_S;
  int32_t dt;                  /* a pigan_dtype value */
  float lambda_pde;            /* weight of the residual penalty (>= 0) */
  float loss_scale;            /* static loss scale (> 0; 1 unless fp16) */
  float lambda_gp;             /* critic gradient penalty weight: 0 for pigan_trunk_step_grads,
                                  >= 0 for pigan_trunk_step_grads_gp */
  int32_t critic_only;         /* 0: every gradient; 1: the critic's update only -- gD, L_D
                                  and L_adv as in the full step; the generators run at the
                                  sensors only (no collocation rows, no residual: L_pde is
                                  reported as 0) and have no reverse pass; their gradient
                                  outputs are neither written nor required (may be NULL) */
} pigan_trunk_desc;

/* Workspace bytes for pigan_trunk_step_grads(_gp) (0 if the descriptor is invalid;
 * includes the penalty's buffers when lambda_gp > 0). */
size_t pigan_trunk_workspace_bytes(const pigan_trunk_desc* s);

/*
 * The training step of pigan_train_step_grads with the shared-trunk generator
 * (same losses, critic and residual; the gradient penalty is
 * pigan_trunk_step_grads_gp).  The trunk is
 * evaluated at the Y sensors (Y head), the u sensors (u head) and the
 * collocation points (jets of both heads).
 *   pT : [G, pigan_trunk_param_count] trunk weights; gT : same shape, the
 *        gradient of L_G = L_adv + L_pde.
 *   pD, gD, z, xc, xsY, xsU, f, f_const, real, w_group, loss, nonfinite, ws,
 *   ws_bytes, stream : as pigan_train_step_grads (device pointers, caller
 *   owned, outputs overwritten, asynchronous on `stream`).
 * Errors: EINVAL for null pointers or invalid shapes (as pigan_train_step_grads),
 * ENOTSUP for unsupported widths or lambda_gp != 0, EWORKSPACE, EDEVICE.
 */
pigan_status pigan_trunk_step_grads(const pigan_trunk_desc* s, const float* pT, const float* pD,
                                    const float* z, const float* xc, const float* xsY,
                                    const float* xsU, const float* f, float f_const,
                                    const float* real, const float* w_group, float* gT, float* gD,
                                    float* loss, int32_t* nonfinite, void* ws, size_t ws_bytes,
                                    void* stream);

/*
 * pigan_trunk_step_grads plus the critic gradient penalty of
 * pigan_train_step_grads_gp (same definition, Sec. I.C and Sec. II.C), the
 * fake snapshot b being the trunk's Y head at the Y sensors and its u head at
 * the u sensors for noise sample b:
 *   gp_eps : [G, min(S, B_r)] fp32 mixing weights (device), required when
 *            lambda_gp > 0 (EINVAL if NULL); gp : [G] fp32 output P_g or NULL.
 * P_g is added to L_D (loss[g][0]) and its gradient to gD; gT is unchanged.
 * Everything else as pigan_trunk_step_grads.
 */
pigan_status pigan_trunk_step_grads_gp(const pigan_trunk_desc* s, const float* pT, const float* pD,
                                       const float* z, const float* xc, const float* xsY,
                                       const float* xsU, const float* f, float f_const,
                                       const float* real, const float* w_group, const float* gp_eps,
                                       float* gT, float* gD, float* loss, float* gp,
                                       int32_t* nonfinite, void* ws, size_t ws_bytes, void* stream);

/*
 * Domain decomposition (Sec. III.B.1): one generator pair for the whole
 * domain and one critic per subdomain of every level of a hierarchy of
 * partitions; critic k is weighted w_k = 1 / (levels x subdomains of its
 * level).  Critic k sees the paper's snapshot of its subdomain,
 *   [Y at the Y sensors idxY[k] | u at the u sensors idxU[k] |
 *    the generated source f = -div(exp(Y) grad u) at the free sensors
 *    idxF[k] (collocation points of the sample) | their coordinates],
 * and real snapshots in the same layout (f = 0 there, their own free-sensor
 * coordinates).  Losses per critic: L_D[k] = w_k (mean D_k(fake) -
 * mean D_k(real)), L_adv[k] = -w_k mean D_k(fake); the generator's loss is
 * sum_k L_adv[k] + L_pde with L_pde = lambda_pde mean r^2 (0 for the paper's
 * purely adversarial form).
 */
typedef struct {
  pigan_mlp genY, genU;        /* n_groups = 1; in_dim = d + n_z */
  pigan_mlp disc;              /* n_groups = D critics; in_dim = mY + mU + nF (1 + d) */
  int32_t d, n_z, S, P;
  int32_t n_sY, n_sU, B_r, chunk_S;
  int32_t mY, mU, nF;          /* inputs of every critic: Y sensors, u sensors, free sensors */
  int32_t dt;                  /* a pigan_dtype value */
  float lambda_pde;            /* >= 0 */
  float loss_scale;            /* > 0 */
  float lambda_gp;             /* critic gradient penalty weight: 0 for pigan_hier_step_grads,
                                  >= 0 for pigan_hier_step_grads_gp */
  int32_t critic_only;         /* 0: every gradient; 1: the critic's update only -- gD and the
                                  losses as in the full step (the critics read the generated
                                  source, so the residual is still evaluated), no reverse pass
                                  of the generator; its gradient outputs are neither written
                                  nor required (may be NULL) */
} pigan_hier_desc;

/* Workspace bytes for pigan_hier_step_grads(_gp) (0 if the descriptor is invalid;
 * includes the penalty's buffers when lambda_gp > 0). */
size_t pigan_hier_workspace_bytes(const pigan_hier_desc* s);

/*
 *   pY, pU : [n_params] generator weights; pD : [D, n_params(disc)] critics.
 *   z, xc, xsY, xsU, f, f_const : as pigan_train_step_grads with G = 1.
 *   idxY : [D, mY], idxU : [D, mU] int32 sensor indices; idxF : [D, nF]
 *          int32 indices into each sample's P collocation points (device).
 *          An index out of range reads zero and sets *nonfinite = 1.
 *   real : [D, B_r, disc in_dim] real snapshots; w_disc : [D] critic weights.
 *   gY, gU : [n_params] gradients of the generator loss; gD : [D, n_params]
 *   gradients of each L_D[k]; loss : [D, 3] = (L_D[k], L_adv[k], L_pde).
 *   nonfinite, ws, ws_bytes, stream : as pigan_train_step_grads.
 * Errors: EINVAL (null pointers, generator n_groups != 1, in_dim mismatch,
 * negative counts), ENOTSUP (widths, lambda_gp != 0), EWORKSPACE, EDEVICE.
 */
pigan_status pigan_hier_step_grads(const pigan_hier_desc* s, const float* pY, const float* pU,
                                   const float* pD, const float* z, const float* xc,
                                   const float* xsY, const float* xsU, const float* f, float f_const,
                                   const int32_t* idxY, const int32_t* idxU, const int32_t* idxF,
                                   const float* real, const float* w_disc, float* gY, float* gU,
                                   float* gD, float* loss, int32_t* nonfinite, void* ws,
                                   size_t ws_bytes, void* stream);

/*
 * pigan_hier_step_grads plus every subdomain critic's gradient penalty, the
 * penalty of pigan_train_step_grads_gp (Sec. I.C, Sec. II.C) taken by each
 * critic of the decomposition (Sec. III.B.1) on its own snapshots:
 *   x_kb = eps_kb real_kb + (1 - eps_kb) F_kb,   b < n_gp = min(S, B_r)
 *          (F_kb: critic k's fake snapshot of noise sample b, all inputs,
 *          the free-sensor coordinates included),
 *   P_k  = w_k lambda_gp mean_b (||grad_v D_k(x_kb)||_2 - 1)^2.
 * P_k is added to L_D[k] (loss[k][0]) and its gradient to gD[k]; gY and gU
 * are unchanged.
 *   gp_eps : [D, n_gp] fp32 mixing weights (device), required when
 *            lambda_gp > 0 (EINVAL if NULL); unused when lambda_gp = 0.
 *   gp     : [D] fp32 output P_k (device) or NULL.
 * Everything else as pigan_hier_step_grads.
 */
pigan_status pigan_hier_step_grads_gp(const pigan_hier_desc* s, const float* pY, const float* pU,
                                      const float* pD, const float* z, const float* xc,
                                      const float* xsY, const float* xsU, const float* f,
                                      float f_const, const int32_t* idxY, const int32_t* idxU,
                                      const int32_t* idxF, const float* real, const float* w_disc,
                                      const float* gp_eps, float* gY, float* gU, float* gD,
                                      float* loss, float* gp, int32_t* nonfinite, void* ws,
                                      size_t ws_bytes, void* stream);

/*
 * Domain decomposition with the shared-trunk generator: the step of
 * pigan_hier_step_grads (same critics, snapshots, weights and losses) with the
 * paper's generator of pigan_trunk_step_grads in place of the pair.  The
 * trunk is evaluated at the Y sensors (Y head), the u sensors (u head) and
 * the collocation points (jets of both heads); the free sensors read the
 * source formed from both heads' jets.
 */
typedef struct {
  pigan_mlp trunk;             /* n_groups = 1; in_dim = d + n_z */
  pigan_mlp disc;              /* n_groups = D critics; in_dim = mY + mU + nF (1 + d) */
  int32_t d, n_z, S, P;
  int32_t n_sY, n_sU, B_r, chunk_S;
  int32_t mY, mU, nF;
  int32_t dt;                  /* a pigan_dtype value */
  float lambda_pde;            /* >= 0 */
  float loss_scale;            /* > 0 */
  float lambda_gp;             /* critic gradient penalty weight: 0 for
                                  pigan_hier_trunk_step_grads, >= 0 for its _gp form */
  int32_t critic_only;         /* 0: every gradient; 1: the critic's update only -- gD and the
                                  losses as in the full step (the critics read the generated
                                  source, so the residual is still evaluated), no reverse pass
                                  of the generator; its gradient outputs are neither written
                                  nor required (may be NULL) */
} pigan_hier_trunk_desc;

/* Workspace bytes for pigan_hier_trunk_step_grads(_gp) (0 if the descriptor is
 * invalid; includes the penalty's buffers when lambda_gp > 0). */
size_t pigan_hier_trunk_workspace_bytes(const pigan_hier_trunk_desc* s);

/*
 *   pT : [pigan_trunk_param_count] trunk weights; gT : same shape, the
 *        gradient of the generator loss sum_k L_adv[k] + L_pde.
 *   pD, z, xc, xsY, xsU, f, f_const, idxY, idxU, idxF, real, w_disc, gD,
 *   loss, nonfinite, ws, ws_bytes, stream : as pigan_hier_step_grads.
 * Errors: as pigan_hier_step_grads (trunk n_groups != 1 is EINVAL).
 */
pigan_status pigan_hier_trunk_step_grads(const pigan_hier_trunk_desc* s, const float* pT,
                                         const float* pD, const float* z, const float* xc,
                                         const float* xsY, const float* xsU, const float* f,
                                         float f_const, const int32_t* idxY, const int32_t* idxU,
                                         const int32_t* idxF, const float* real,
                                         const float* w_disc, float* gT, float* gD, float* loss,
                                         int32_t* nonfinite, void* ws, size_t ws_bytes,
                                         void* stream);

/*
 * pigan_hier_trunk_step_grads plus every subdomain critic's gradient penalty,
 * as pigan_hier_step_grads_gp (gp_eps [D, min(S, B_r)], gp [D] or NULL; gT
 * unchanged by the penalty).
 */
pigan_status pigan_hier_trunk_step_grads_gp(const pigan_hier_trunk_desc* s, const float* pT,
                                            const float* pD, const float* z, const float* xc,
                                            const float* xsY, const float* xsU, const float* f,
                                            float f_const, const int32_t* idxY,
                                            const int32_t* idxU, const int32_t* idxF,
                                            const float* real, const float* w_disc,
                                            const float* gp_eps, float* gT, float* gD, float* loss,
                                            float* gp, int32_t* nonfinite, void* ws,
                                            size_t ws_bytes, void* stream);

/*
 * pigan_adam_update — one update of fp32 master weights from the fp32
 * gradients of a training step (the paper keeps single-precision master
 * weights and adaptive loss scaling, Sec. III.C; it names no optimizer, so
 * the update is Adam in its textbook form):
 *   m = beta1 m + (1 - beta1) g,  v = beta2 v + (1 - beta2) g^2,
 *   p = p - lr (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps).
 *   n      : number of parameters (>= 0);
 *   params, m, v : [n] fp32 device arrays, updated in place (m, v start at 0);
 *   grads  : [n] fp32 device gradients (already divided by the loss scale);
 *   t      : 1-based count of updates including this one;
 *   skip   : device int32 (the step's `nonfinite` flag) or NULL; when it
 *            holds a non-zero value the launch leaves params, m and v
 *            unchanged (decided on the device, no host synchronisation).
 * Asynchronous on `stream`.  EINVAL for null arrays (n > 0), t < 1, betas
 * outside [0, 1), non-finite lr or negative eps; EDEVICE on launch failure.
 */
pigan_status pigan_adam_update(int64_t n, float* params, const float* grads, float* m, float* v,
                               float lr, float beta1, float beta2, float eps, int32_t t,
                               const int32_t* skip, void* stream);

/* Thread-local description of the last non-OK status ("" if none). */
const char* pigan_last_error(void);

/*
 * Kernel timing (instrumentation, not part of the method).  While enabled,
 * every library kernel launch is bracketed by HIP events recorded on the
 * caller's stream, and its algorithmic work is recorded with it.
 * pigan_profile_read() must be called after the caller has synchronised the
 * stream; it aggregates per kernel family and resets the record.
 */
typedef struct {
  char name[48];          /* kernel family, e.g. "gemm_fwd" */
  int64_t launches;
  double total_ms;        /* sum of event-measured durations */
  double flops;           /* algorithmic matrix FLOPs of all launches (2*M*N*K) */
  double bytes;           /* algorithmic HBM bytes of all launches */
} pigan_kernel_stat;

pigan_status pigan_profile_enable(int32_t on);
pigan_status pigan_profile_read(pigan_kernel_stat* out, int32_t max_entries, int32_t* n_entries);

#ifdef __cplusplus
}
#endif

#endif /* PIGAN_H */
