// Memory-bound kernels of the PI-GAN step for gfx950: the generator's first
// layer (z-projection hoisted per sample, derivative seeds are columns of
// W1), the scalar output layer, the Darcy residual and its cotangents, the
// output-layer reverse pass, the first-layer weight gradient, discriminator
// score cotangents, losses, weight casts.  All reductions are fixed-order
// (partial sums per block, then an ordered sum), never atomics.
#include "pointwise.h"

namespace pigan {

// ---------------------------------------------------------------------------
// zp[g][s][n] = b1[n] + sum_j W1[n][d + j] z[g][s][j]   (summed in fp64,
// stored in fp32)
// ---------------------------------------------------------------------------
__global__ void k_zproj(const float* __restrict__ p1, int64_t p_g, int in_dim, int d, int W,
                        const float* __restrict__ z, int64_t z_g, int n_z, int S, float* __restrict__ zp,
                        int64_t zp_g) {
  const int g = blockIdx.z;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)S * W) return;
  const int s = (int)(idx / W), n = (int)(idx % W);
  const float* Wn = p1 + g * p_g + (int64_t)n * in_dim + d;
  const float* zs = z + g * z_g + (int64_t)s * n_z;
  double a = (double)p1[g * p_g + (int64_t)W * in_dim + n];
  for (int j = 0; j < n_z; ++j) a += (double)Wn[j] * (double)zs[j];
  zp[g * zp_g + idx] = (float)a;
}

// ---------------------------------------------------------------------------
// 8-wide vector access in the storage type (16 bytes in bf16/fp16, 32 in fp32)
// ---------------------------------------------------------------------------
template <class T>
__device__ __forceinline__ void load8(const T* p, float* v) {
  if (sizeof(T) == 2) {
    const uint4 raw = *(const uint4*)p;
    const T* e = (const T*)&raw;
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = Elem<T>::to_f(e[i]);
  } else {
    const float4 a = *(const float4*)p, b = *((const float4*)p + 1);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}

template <class T>
__device__ __forceinline__ void store8(T* p, const float* v) {
  if (sizeof(T) == 2) {
    uint4 raw;
    T* e = (T*)&raw;
#pragma unroll
    for (int i = 0; i < 8; ++i) e[i] = Elem<T>::from_f(v[i]);
    *(uint4*)p = raw;
  } else {
    *(float4*)p = make_float4(v[0], v[1], v[2], v[3]);
    *((float4*)p + 1) = make_float4(v[4], v[5], v[6], v[7]);
  }
}

// ---------------------------------------------------------------------------
// first layer: a = zp[s] + W1[:, :d] x ; a'_i = W1[:, i] ; a''_i = 0
// one thread per (point, 8 columns)
// ---------------------------------------------------------------------------
// A thread keeps one group of 8 columns (and its x-part weights, loaded once)
// and walks FF_PPB points of the block, PPI = 256 / (W / 8) at a time; stores
// leave as full 16-byte pieces of consecutive columns.
constexpr int FF_PPB = 32;

template <class T, int ND1, int ND2, bool X64 = false>
__global__ void __launch_bounds__(256)
k_first_fwd(FirstArgs<T> p) {
  constexpr int C = 1 + ND1 + ND2;
  const int g = blockIdx.z;
  const int G8 = p.W / 8;
  const int TPP = G8 < 256 ? G8 : 256;   // threads per point
  const int PPI = 256 / TPP;             // points per iteration
  const int cg0 = threadIdx.x % TPP;
  const int64_t pbeg = (int64_t)blockIdx.x * FF_PPB;
  int64_t pend = pbeg + FF_PPB;
  if (pend > p.seg.n_points) pend = p.seg.n_points;
  const int64_t pl = p.seg.plane * p.ldo;
  for (int cg = cg0; cg < G8; cg += TPP) {
    const int n0 = cg * 8;
    const float* W1 = p.p1 + g * p.p_g + (int64_t)n0 * p.in_dim;
    float wc[3][8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
      for (int i = 0; i < 3; ++i) wc[i][e] = i < p.d ? W1[(int64_t)e * p.in_dim + i] : 0.0f;
    for (int64_t pt = pbeg + threadIdx.x / TPP; pt < pend; pt += PPI) {
      const int64_t s = pt / p.Pn;
      const int64_t xr = p.x_shared ? pt % p.Pn : pt;
      const float* xv = p.x + g * p.x_g + xr * p.d;
      float x[3] = {0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int i = 0; i < 3; ++i)
        if (i < p.d) x[i] = xv[i];
      float a[8];
      load8<float>(p.zp + g * p.zp_g + s * p.W + n0, a);
#pragma unroll
      for (int e = 0; e < 8; ++e)
#pragma unroll
        for (int i = 0; i < 3; ++i) a[e] += wc[i][e] * x[i];
      float h[C][8];
      float s8[8], sp8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float t, sd;
        tanh_pair<X64>(a[e], t, sd);
        h[0][e] = t;
        s8[e] = sd;
        sp8[e] = -2.0f * t * sd;
      }
#pragma unroll
      for (int i = 0; i < ND1; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e) h[1 + i][e] = s8[e] * wc[i][e];
#pragma unroll
      for (int i = 0; i < ND2; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e) h[1 + ND1 + i][e] = sp8[e] * wc[i][e] * wc[i][e];
      const int64_t base = g * p.o_g + (p.seg.row0 + pt) * p.ldo + n0;
      if (p.out_a) {
        store8<T>(p.out_a + base, a);
#pragma unroll
        for (int i = 0; i < ND1; ++i) store8<T>(p.out_a + base + (1 + i) * pl, wc[i]);
        float z8[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
        for (int i = 0; i < ND2; ++i) store8<T>(p.out_a + base + (1 + ND1 + i) * pl, z8);
      }
#pragma unroll
      for (int k = 0; k < C; ++k) store8<T>(p.out_h + base + k * pl, h[k]);
    }
  }
}

// ---------------------------------------------------------------------------
// scalar output layer: y[row] = w_out . H[row] (+ b_out on value rows)
// eight lanes per row, 16-byte loads, shuffle reduction; fp32 storage (the
// sensor rows and the critic) sums in fp64
// ---------------------------------------------------------------------------
template <class T>
__global__ void __launch_bounds__(256)
k_out_fwd(const T* __restrict__ H, int64_t h_g, int64_t ldh, int64_t R, int64_t n_value, int W,
          const float* __restrict__ wout, int64_t w_g, float* __restrict__ y, int64_t y_g) {
  constexpr int EPP = 16 / (int)sizeof(T);
  const int g = blockIdx.z;
  const int team = threadIdx.x >> 3, e = threadIdx.x & 7;
  const int64_t row = (int64_t)blockIdx.x * 32 + team;
  typedef typename std::conditional<sizeof(T) == 4, double, float>::type Acc;
  const float* w = wout + g * w_g;
  Acc acc = 0;
  if (row < R) {
    const T* hr = H + g * h_g + row * ldh;
    for (int c = e * EPP; c < W; c += 8 * EPP) {
      uint4 v = *(const uint4*)(hr + c);
      const T* hv = (const T*)&v;
#pragma unroll
      for (int q = 0; q < EPP; ++q) acc += (Acc)w[c + q] * (Acc)Elem<T>::to_f(hv[q]);
    }
  }
  acc += __shfl_xor(acc, 1);
  acc += __shfl_xor(acc, 2);
  acc += __shfl_xor(acc, 4);
  if (row < R && e == 0) y[g * y_g + row] = (float)(acc + (row < n_value ? (Acc)w[W] : (Acc)0));
}

// ---------------------------------------------------------------------------
// Darcy residual r = -exp(Y)(sum_i dY_i dU_i + sum_i ddU_i) - f  and the
// cotangents of L_pde = w lambda mean r^2 with respect to the jets:
//   q = 2 w lambda r / (S P);   gY = q (r + f);  g dY_i = -q e^Y dU_i;
//   g dU_i = -q e^Y dY_i;  g ddU_i = -q e^Y;  g U = 0.
// Per-block partial sums of r^2 (double) for the loss.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256)
k_residual(ResidArgs p) {
  __shared__ double red[256];
  const int g = blockIdx.z;
  const int64_t pt = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  double r2 = 0.0;
  if (pt < p.M) {
    const float* jy = p.jY + g * p.jy_g + p.offY;
    const float* ju = p.jU + g * p.ju_g + p.offU;
    const float Y = jy[pt];
    const float f = p.f ? p.f[g * p.f_g + pt] : p.f_const;
    float flux = 0.0f;
    for (int i = 0; i < p.d; ++i) flux += jy[(1 + i) * p.plane + pt] * ju[(1 + i) * p.plane + pt];
    for (int i = 0; i < p.d; ++i) flux += ju[(1 + p.d + i) * p.plane + pt];
    const float eY = expf(Y);
    const float r = -eY * flux - f;
    if (p.r) p.r[g * p.r_g + pt] = r;
    r2 = (double)r * (double)r;
    if (p.gY) {
      const float w = p.w_group ? p.w_group[g] : 1.0f;
      const float q = p.qscale * w * r + (p.gq ? p.gq[g * p.gq_g + pt] : 0.0f);
      float* gy = p.gY + g * p.jy_g + p.offY;
      float* gu = p.gU + g * p.ju_g + p.offU;
      gy[pt] = q * (r + f);
      gu[pt] = 0.0f;
      for (int i = 0; i < p.d; ++i) {
        gy[(1 + i) * p.plane + pt] = -q * eY * ju[(1 + i) * p.plane + pt];
        gu[(1 + i) * p.plane + pt] = -q * eY * jy[(1 + i) * p.plane + pt];
        gu[(1 + p.d + i) * p.plane + pt] = -q * eY;
      }
    }
  }
  if (p.part) {
    red[threadIdx.x] = r2;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
      if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
      __syncthreads();
    }
    if (threadIdx.x == 0) p.part[(int64_t)g * gridDim.x + blockIdx.x] = red[0];
  }
}

// acc[g*stride + slot] += sum_b part[g][b]   (one block per group, fixed order)
__global__ void __launch_bounds__(256)
k_sum_partials(const double* __restrict__ part, int nb, double* acc, int acc_stride, int slot) {
  __shared__ double red[256];
  const int g = blockIdx.x;
  double s = 0.0;
  for (int b = threadIdx.x; b < nb; b += 256) s += part[(int64_t)g * nb + b];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) acc[g * acc_stride + slot] += red[0];
}

// ---------------------------------------------------------------------------
// discriminator input rows: fake snapshots [Y sensors | u sensors] from the
// generator outputs (b < n_fake), then real snapshots; zero padded to ldx.
// ---------------------------------------------------------------------------
template <class T>
__global__ void k_snap_fill(const float* __restrict__ yY, int64_t yY_g, const float* __restrict__ yU,
                            int64_t yU_g, int nY, int nU, int ldY, int ldU, int offU, int n_fake,
                            const float* __restrict__ real, int64_t real_g, int n_real, int n_in, T* __restrict__ X,
                            int64_t x_g, int ldx) {
  const int g = blockIdx.z;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int B = n_fake + n_real;
  if (idx >= (int64_t)B * ldx) return;
  const int b = (int)(idx / ldx), j = (int)(idx % ldx);
  float v = 0.0f;
  if (j < n_in) {
    if (b < n_fake) {
      v = j < nY ? yY[g * yY_g + (int64_t)b * ldY + j] : yU[g * yU_g + (int64_t)b * ldU + offU + (j - nY)];
    } else {
      v = real[g * real_g + (int64_t)(b - n_fake) * n_in + j];
    }
  }
  X[g * x_g + idx] = Elem<T>::from_f(v);
}

// ---------------------------------------------------------------------------
// Critic gradient penalty (WGAN-GP member of the critic family the paper
// cites): interpolates x_b = eps_b R_b + (1 - eps_b) F_b of the n pairs of a
// chunk (fake row i is the chunk's sample i, global pair b = b0 + i), stored
// in the discriminator's input rows [0, n) in the storage type.
// ---------------------------------------------------------------------------
template <class T>
__global__ void k_gp_mix(const float* __restrict__ yY, int64_t yY_g, const float* __restrict__ yU, int64_t yU_g,
                         int nY, int nU, int ldY, int ldU, int offU, const float* __restrict__ real, int64_t real_g,
                         const float* __restrict__ eps, int64_t eps_g, int b0, int n, int n_in, T* __restrict__ X,
                         int64_t x_g, int ldx) {
  const int g = blockIdx.z;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)n * ldx) return;
  const int i = (int)(idx / ldx), j = (int)(idx % ldx);
  float v = 0.0f;
  if (j < n_in) {
    const float f = j < nY ? yY[g * yY_g + (int64_t)i * ldY + j] : yU[g * yU_g + (int64_t)i * ldU + offU + (j - nY)];
    const float r = real[g * real_g + (int64_t)(b0 + i) * n_in + j];
    const float e = eps[g * eps_g + b0 + i];
    v = e * r + (1.0f - e) * f;
  }
  X[g * x_g + idx] = Elem<T>::from_f(v);
}

// seeds [0, n) = v0, [n, 2n) = v1 (fp32), one group per grid z
__global__ void k_fill2(float* __restrict__ seed, int64_t s_g, int n, float v0, float v1, int two) {
  const int g = blockIdx.z;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) seed[g * s_g + i] = v0;
  if (two && i < n) seed[g * s_g + n + i] = v1;
}

// One block per pair row: norm of the critic's input gradient g_i, the
// penalty term (|g_i| - 1)^2 (double, per row; summed later in row order),
// and the tangent row c_i = scale (|g_i| - 1)/|g_i| g_i stored as input row
// n + i (zero for g_i = 0, which has no gradient direction).
template <class T>
__global__ void __launch_bounds__(256)
k_gp_norm(const float* __restrict__ gin, int64_t g_g, int n, int n_in, const float* __restrict__ w_group,
          float scale, double* __restrict__ part, int64_t p_g, T* __restrict__ X, int64_t x_g, int ldx) {
  __shared__ double red[256];
  const int g = blockIdx.z;
  const int i = blockIdx.x;
  const float* gi = gin + g * g_g + (int64_t)i * n_in;
  double acc = 0.0;
  for (int j = threadIdx.x; j < n_in; j += 256) acc += (double)gi[j] * (double)gi[j];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int h = 128; h > 0; h >>= 1) {
    if ((int)threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
    __syncthreads();
  }
  const double nrm = sqrt(red[0]);
  if (threadIdx.x == 0) part[g * p_g + i] = (nrm - 1.0) * (nrm - 1.0);
  const float w = w_group ? w_group[g] : 1.0f;
  const float coef = nrm > 0.0 ? (float)((nrm - 1.0) / nrm) * scale * w : 0.0f;
  T* xr = X + g * x_g + (int64_t)(n + i) * ldx;
  for (int j = threadIdx.x; j < ldx; j += 256) xr[j] = Elem<T>::from_f(j < n_in ? coef * gi[j] : 0.0f);
}

// ---------------------------------------------------------------------------
// critic cotangents and score sums (one block per group):
//   dL_D/dD(fake_s) = w/S,  dL_D/dD(real_b) = -w/B_r   (times the loss scale)
//   acc[g][0] += sum D(fake), acc[g][1] += sum D(real)
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256)
k_disc_seed(const float* __restrict__ score, int64_t sc_g, int n_fake, int n_real, int S_total, int B_total,
            const float* __restrict__ w_group, float loss_scale, float* __restrict__ seed, double* acc,
            int acc_stride) {
  __shared__ double red[2][256];
  const int g = blockIdx.x;
  const float w = w_group ? w_group[g] : 1.0f;
  double sf = 0.0, sr = 0.0;
  for (int b = threadIdx.x; b < n_fake + n_real; b += 256) {
    const float v = score[g * sc_g + b];
    if (b < n_fake) {
      sf += v;
      seed[g * sc_g + b] = loss_scale * w / (float)S_total;
    } else {
      sr += v;
      seed[g * sc_g + b] = -loss_scale * w / (float)B_total;
    }
  }
  red[0][threadIdx.x] = sf;
  red[1][threadIdx.x] = sr;
  __syncthreads();
  for (int k = 128; k > 0; k >>= 1) {
    if ((int)threadIdx.x < k) {
      red[0][threadIdx.x] += red[0][threadIdx.x + k];
      red[1][threadIdx.x] += red[1][threadIdx.x + k];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    acc[g * acc_stride + 0] += red[0][0];
    acc[g * acc_stride + 1] += red[1][0];
  }
}

// ---------------------------------------------------------------------------
// output layer reverse pass for one segment of points:
//   dH_k[pt][n] = gbar_k[pt] w_out[n]  -> carry reverse with the saved A_L
//   partial dw_out[n] = sum gbar_k h_k (h re-formed from A_L),
//   partial db_out   = sum over value rows of gbar_0.
// A thread owns 8 consecutive columns; TPP = W/8 (<= 256) threads per point,
// 256/TPP points per pass; up to two column groups per thread (W <= 4096).
// Partials are fp64: part[g][slot][W+1].
// ---------------------------------------------------------------------------
template <class T, int ND1, int ND2, bool X64 = false>
__global__ void __launch_bounds__(256)
k_out_bwd(OutBwdArgs<T> p) {
  constexpr int C = 1 + ND1 + ND2;
  __shared__ double red[256 * 8];
  const int g = blockIdx.z;
  const int W = p.W;
  const int G8 = W / 8;
  const int TPP = G8 < 256 ? G8 : 256;
  const int PPP = 256 / TPP;
  const int lt = threadIdx.x % TPP;
  const int lp = threadIdx.x / TPP;
  const int64_t pbeg = (int64_t)blockIdx.x * p.ppb;
  int64_t pend = pbeg + p.ppb;
  if (pend > p.seg.n_points) pend = p.seg.n_points;
  const float* w = p.wout + g * p.w_g;
  const float* gb = p.gbar + g * p.gb_g;
  double dw[2][8];
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int e = 0; e < 8; ++e) dw[c][e] = 0.0;
  double db = 0.0;
  const int64_t pl = p.seg.plane * p.ldo;
  for (int64_t pt = pbeg + lp; pt < pend; pt += PPP) {
    float gk[C];
#pragma unroll
    for (int k = 0; k < C; ++k) gk[k] = gb[p.seg.row0 + k * p.seg.plane + pt];
    if (lt == 0) db += gk[0];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int cg = lt + 256 * c;
      if (cg >= G8) continue;
      const int n0 = cg * 8;
      float wn[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) wn[e] = w[n0 + e];   // parameter vectors are only 4-byte aligned
      const int64_t base = g * p.o_g + (p.seg.row0 + pt) * p.ldo + n0;
      float ap[C][8];
#pragma unroll
      for (int k = 0; k < C; ++k) load8<T>(p.A + base + k * pl, ap[k]);
      float da[C][8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float t, s;
        tanh_pair<X64>(ap[0][e], t, s);
        const float sp = -2.0f * t * s;
        const float spp = 2.0f * s * (3.0f * t * t - 1.0f);
        float hsum = gk[0] * t;
#pragma unroll
        for (int i = 0; i < ND1; ++i) hsum += gk[1 + i] * s * ap[1 + i][e];
#pragma unroll
        for (int i = 0; i < ND2; ++i)
          hsum += gk[1 + ND1 + i] * (s * ap[1 + ND1 + i][e] + sp * ap[1 + i][e] * ap[1 + i][e]);
        dw[c][e] += (double)hsum;
        float ga = s * gk[0];
#pragma unroll
        for (int i = 0; i < ND1; ++i) ga += sp * ap[1 + i][e] * gk[1 + i];
#pragma unroll
        for (int i = 0; i < ND2; ++i) ga += (sp * ap[1 + ND1 + i][e] + spp * ap[1 + i][e] * ap[1 + i][e]) * gk[1 + ND1 + i];
        da[0][e] = ga * wn[e];
#pragma unroll
        for (int i = 0; i < ND1; ++i) {
          float gd = s * gk[1 + i];
          if (i < ND2) gd += 2.0f * sp * ap[1 + i][e] * gk[1 + ND1 + i];
          da[1 + i][e] = gd * wn[e];
        }
#pragma unroll
        for (int i = 0; i < ND2; ++i) da[1 + ND1 + i][e] = s * gk[1 + ND1 + i] * wn[e];
      }
#pragma unroll
      for (int k = 0; k < C; ++k) store8<T>(p.dA + base + k * pl, da[k]);
    }
  }
  // block reduction over the PPP point lanes, fixed order, fp64
  double* pw = p.part + ((int64_t)g * p.n_slots + p.slot0 + blockIdx.x) * (W + 1);
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    if (G8 <= 256 * c) continue;
#pragma unroll
    for (int e = 0; e < 8; ++e) red[threadIdx.x * 8 + e] = dw[c][e];
    __syncthreads();
    const int cg = lt + 256 * c;
    if (lp == 0 && cg < G8) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        double s = 0.0;
        for (int q = 0; q < PPP; ++q) s += red[(q * TPP + lt) * 8 + e];
        pw[cg * 8 + e] = s;
      }
    }
    __syncthreads();
  }
  red[threadIdx.x] = db;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int q = 0; q < PPP; ++q) s += red[q * TPP];
    pw[W] = s;
  }
}

// ---------------------------------------------------------------------------
// Output layer of a shared trunk, reverse pass: two linear heads (Y, u) on the
// last trunk activations h_L.  Per point and stream k the activation cotangent
// is g_h_k = w_Y gY_k + w_u gu_k; the head weight gradients are sums over rows
// of g_k h_k (h_L read as stored: with a residual block on top it is not
// tanh(a_L)), the bias gradients sums of the value cotangents.  g_h is stored
// (for the skip below the top block) when p.gh is set, then carried back
// through tanh into dA.  fp64 per-block partials [2 (W + 1)], fixed order.
// ---------------------------------------------------------------------------
template <class T, int ND1, int ND2, bool X64 = false>
__global__ void __launch_bounds__(256)
k_out2_bwd(Out2BwdArgs<T> p) {
  constexpr int C = 1 + ND1 + ND2;
  __shared__ double red[256 * 8];
  const int g = blockIdx.z;
  const int W = p.W;
  const int G8 = W / 8;
  const int TPP = G8 < 256 ? G8 : 256;
  const int PPP = 256 / TPP;
  const int lt = threadIdx.x % TPP;
  const int lp = threadIdx.x / TPP;
  const int64_t pbeg = (int64_t)blockIdx.x * p.ppb;
  int64_t pend = pbeg + p.ppb;
  if (pend > p.seg.n_points) pend = p.seg.n_points;
  const float* w0 = p.wout + g * p.w_g;
  const float* w1 = w0 + W + 1;
  const float* gb0 = p.gbar0 + g * p.gb_g;
  const float* gb1 = p.gbar1 + g * p.gb_g;
  double dw[2][2][8];
#pragma unroll
  for (int hd = 0; hd < 2; ++hd)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int e = 0; e < 8; ++e) dw[hd][c][e] = 0.0;
  double db0 = 0.0, db1 = 0.0;
  const int64_t pl = p.seg.plane * p.ldo;
  for (int64_t pt = pbeg + lp; pt < pend; pt += PPP) {
    float g0[C], g1[C];
#pragma unroll
    for (int k = 0; k < C; ++k) {
      g0[k] = gb0[p.seg.row0 + k * p.seg.plane + pt];
      g1[k] = gb1[p.seg.row0 + k * p.seg.plane + pt];
    }
    if (lt == 0) {
      db0 += g0[0];
      db1 += g1[0];
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int cg = lt + 256 * c;
      if (cg >= G8) continue;
      const int n0 = cg * 8;
      float wa[8], wb[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        wa[e] = w0[n0 + e];   // parameter vectors are only 4-byte aligned
        wb[e] = w1[n0 + e];
      }
      const int64_t base = g * p.o_g + (p.seg.row0 + pt) * p.ldo + n0;
      float gh[C][8];
#pragma unroll
      for (int k = 0; k < C; ++k) {
        float hv[8];
        load8<T>(p.H + base + k * pl, hv);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          dw[0][c][e] += (double)(g0[k] * hv[e]);
          dw[1][c][e] += (double)(g1[k] * hv[e]);
          gh[k][e] = wa[e] * g0[k] + wb[e] * g1[k];
        }
      }
      if (p.gh) {
#pragma unroll
        for (int k = 0; k < C; ++k) store8<T>(p.gh + base + k * pl, gh[k]);
      }
      float ap[C][8];
#pragma unroll
      for (int k = 0; k < C; ++k) load8<T>(p.A + base + k * pl, ap[k]);
      float da[C][8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float t, s;
        tanh_pair<X64>(ap[0][e], t, s);
        const float sp = -2.0f * t * s;
        const float spp = 2.0f * s * (3.0f * t * t - 1.0f);
        float ga = s * gh[0][e];
#pragma unroll
        for (int i = 0; i < ND1; ++i) ga += sp * ap[1 + i][e] * gh[1 + i][e];
#pragma unroll
        for (int i = 0; i < ND2; ++i)
          ga += (sp * ap[1 + ND1 + i][e] + spp * ap[1 + i][e] * ap[1 + i][e]) * gh[1 + ND1 + i][e];
        da[0][e] = ga;
#pragma unroll
        for (int i = 0; i < ND1; ++i) {
          float gd = s * gh[1 + i][e];
          if (i < ND2) gd += 2.0f * sp * ap[1 + i][e] * gh[1 + ND1 + i][e];
          da[1 + i][e] = gd;
        }
#pragma unroll
        for (int i = 0; i < ND2; ++i) da[1 + ND1 + i][e] = s * gh[1 + ND1 + i][e];
      }
#pragma unroll
      for (int k = 0; k < C; ++k) store8<T>(p.dA + base + k * pl, da[k]);
    }
  }
  // block reduction over the PPP point lanes, fixed order, fp64
  double* pw = p.part + ((int64_t)g * p.n_slots + p.slot0 + blockIdx.x) * 2 * (W + 1);
#pragma unroll
  for (int hd = 0; hd < 2; ++hd) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      if (G8 <= 256 * c) continue;
#pragma unroll
      for (int e = 0; e < 8; ++e) red[threadIdx.x * 8 + e] = dw[hd][c][e];
      __syncthreads();
      const int cg = lt + 256 * c;
      if (lp == 0 && cg < G8) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          double sm = 0.0;
          for (int q = 0; q < PPP; ++q) sm += red[(q * TPP + lt) * 8 + e];
          pw[hd * (W + 1) + cg * 8 + e] = sm;
        }
      }
      __syncthreads();
    }
    red[threadIdx.x] = hd == 0 ? db0 : db1;
    __syncthreads();
    if (threadIdx.x == 0) {
      double sm = 0.0;
      for (int q = 0; q < PPP; ++q) sm += red[q * TPP];
      pw[hd * (W + 1) + W] = sm;
    }
    __syncthreads();
  }
}

// rows [0, na) of a then [0, nb) of b, d floats each, per group
__global__ void k_concat_rows(const float* __restrict__ a, int64_t a_g, int na, const float* __restrict__ b,
                              int64_t b_g, int nb, int d, float* __restrict__ out, int64_t o_g) {
  const int g = blockIdx.z;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)(na + nb) * d) return;
  const int64_t row = i / d, c = i % d;
  out[g * o_g + i] = row < na ? a[g * a_g + row * d + c] : b[g * b_g + (row - na) * d + c];
}

__global__ void k_fill_f32(float* __restrict__ p, int64_t n, int64_t p_g, float v) {
  const int g = blockIdx.z;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[g * p_g + i] = v;
}

// ---------------------------------------------------------------------------
// Domain decomposition (one critic per subdomain, grid z = critic k).  Fake
// row b (sample b of the chunk) of critic k's snapshot: [Y at sensors
// idxY[k] | u at sensors idxU[k] | the generated source N = r + f at the free
// sensors idxF[k] (collocation points of the sample) | their coordinates];
// real rows follow.  Indices out of range read zero and raise h.bad.  The
// sensor rows of sample b sit at b * ldY (Y) and b * ldU + offU (u): a
// generator pair keeps them in separate arrays, the shared trunk in one row
// block per sample ([Y sensors ; u sensors], Y head and u head arrays).
// With eps set (and no real rows) fake row b becomes the gradient penalty's
// interpolate of pair b0 + b: eps R + (1 - eps) F with R that pair's real
// snapshot of critic k and eps = eps[k][b0 + b].
// ---------------------------------------------------------------------------
template <class T>
__global__ void k_hier_snap(HierSnap h, int n_fake, const float* __restrict__ real, int64_t real_g, int n_real,
                            T* __restrict__ X, int64_t x_g, int ldx, const float* __restrict__ eps, int64_t eps_g,
                            int b0) {
  const int k = blockIdx.z;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)(n_fake + n_real) * ldx) return;
  const int b = (int)(idx / ldx), j = (int)(idx % ldx);
  float v = 0.0f;
  if (j < h.n_in) {
    if (b < n_fake) {
      const int e1 = h.mY, e2 = e1 + h.mU, e3 = e2 + h.nF;
      if (j < e1) {
        const int i = h.idxY[(int64_t)k * h.mY + j];
        if (i >= 0 && i < h.nsY) v = h.jY[(int64_t)b * h.ldY + i];
        else *h.bad = 1;
      } else if (j < e2) {
        const int i = h.idxU[(int64_t)k * h.mU + (j - e1)];
        if (i >= 0 && i < h.nsU) v = h.jU[(int64_t)b * h.ldU + h.offU + i];
        else *h.bad = 1;
      } else {
        const int q = j < e3 ? j - e2 : (j - e3) / h.d;
        const int i = h.idxF[(int64_t)k * h.nF + q];
        if (i >= 0 && i < h.P) {
          const int64_t pt = (int64_t)b * h.P + i;
          v = j < e3 ? h.r[pt] + (h.f ? h.f[pt] : h.f_const) : h.xc[pt * h.d + (j - e3) % h.d];
        } else {
          *h.bad = 1;
        }
      }
      if (eps) {   // penalty interpolate of the pair b0 + b
        const float e = eps[k * eps_g + b0 + b];
        v = e * real[k * real_g + (int64_t)(b0 + b) * h.n_in + j] + (1.0f - e) * v;
      }
    } else {
      v = real[k * real_g + (int64_t)(b - n_fake) * h.n_in + j];
    }
  }
  X[k * x_g + idx] = Elem<T>::from_f(v);
}

// One block per sample b.  Its targets -- Y sensors, u sensors, then the
// sample's collocation points -- are owned round-robin by the threads (slot t
// of a tile by thread t % HS_NTH).  The critic inputs of one index list are
// staged through LDS in chunks (target and cotangent of each input, in the
// order critic k, then input j); every thread then walks the chunk and adds
// the inputs read from its own targets into its LDS slots, so each target
// accumulates in (k, j) order and no two threads touch one slot.  The cost is
// one pass over the inputs per tile of targets, whatever the number of
// critics.  Coordinates carry no cotangent.
constexpr int HS_TILE = 8192, HS_NTH = 256, HS_CHUNK = 2048;

__global__ void __launch_bounds__(HS_NTH)
k_hier_scatter(HierSnap h, const float* __restrict__ dX, int64_t dx_g, int ldx, int D, float* __restrict__ gY,
               float* __restrict__ gU, float* __restrict__ gN) {
  __shared__ float acc[HS_TILE];
  __shared__ __attribute__((aligned(16))) int etgt[HS_CHUNK];
  __shared__ __attribute__((aligned(16))) float eval[HS_CHUNK];
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const float* row = dX + (int64_t)b * ldx;
  const int nT = h.nsY + h.nsU + h.P;
  auto target = [&](int t) -> float* {
    if (t < h.nsY) return gY + (int64_t)b * h.ldY + t;
    if (t < h.nsY + h.nsU) return gU + (int64_t)b * h.ldU + h.offU + (t - h.nsY);
    return gN + (int64_t)b * h.P + (t - h.nsY - h.nsU);
  };
  for (int t0 = 0; t0 < nT; t0 += HS_TILE) {
    const int len = t0 + HS_TILE < nT ? HS_TILE : nT - t0;
    for (int t = tid; t < len; t += HS_NTH) acc[t] = *target(t0 + t);
    // inputs of list `idx` (m per critic, columns col0.. of the rows) read
    // from targets base + i, i in [0, n)
    auto pass = [&](const int32_t* __restrict__ idx, int m, int col0, int n, int base) {
      const int total = D * m;
      for (int c0 = 0; c0 < total; c0 += HS_CHUNK) {
        const int cnt = c0 + HS_CHUNK < total ? HS_CHUNK : total - c0;
        __syncthreads();                           // the previous chunk is consumed
        for (int q = tid; q < cnt; q += HS_NTH) {
          const int e = c0 + q, k = e / m, j = e - k * m;
          const int i = idx[e];
          etgt[q] = (i >= 0 && i < n) ? base + i - t0 : -1;
          eval[q] = row[k * dx_g + col0 + j];
        }
        for (int q = cnt + tid; q < ((cnt + 3) & ~3); q += HS_NTH) etgt[q] = -1;   // pad to a multiple of 4
        __syncthreads();
        // four inputs per LDS read (all lanes read the same words), several reads in flight
#pragma unroll 4
        for (int q = 0; q < cnt; q += 4) {
          const int4 t4 = *(const int4*)(etgt + q);
          const float4 v4 = *(const float4*)(eval + q);
          const int tt[4] = {t4.x, t4.y, t4.z, t4.w};
          const float vv[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int t = tt[u];
            if (t >= 0 && t < len && (t & (HS_NTH - 1)) == tid) acc[t] += vv[u];
          }
        }
      }
    };
    pass(h.idxY, h.mY, 0, h.nsY, 0);
    pass(h.idxU, h.mU, h.mY, h.nsU, h.nsY);
    pass(h.idxF, h.nF, h.mY + h.mU, h.P, h.nsY + h.nsU);
    for (int t = tid; t < len; t += HS_NTH) *target(t0 + t) = acc[t];
    __syncthreads();                               // before the next tile's staging
  }
}

__global__ void k_hier_pde_loss(const double* __restrict__ acc, int slot, float lambda_pde, int64_t SP, float* loss,
                                int D, int32_t* nonfinite) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= D) return;
  const double Lp = (double)lambda_pde * acc[slot] / (double)SP;
  loss[3 * k + 2] = (float)Lp;
  if (k == 0 && !__builtin_isfinite(Lp)) *nonfinite = 1;
}

// ---------------------------------------------------------------------------
// dst (+)= scale * sum over slots of part[g][slot][col], fp64, fixed order.
// A block is 256 / SG column lanes x SG slot groups (SG = 1, 8, 32 or 128); group q sums slots q,
// q + SG, ... and the SG group sums are combined by a fixed pairwise tree.
// Column col maps to dst[(col / Jp) * J + col % Jp] and is skipped when
// col % Jp >= J (padding).  VEC consecutive columns per lane (VEC = 4: one
// 16-byte load per slot); the per-column summation order depends on SG only.
// Few columns take many slot groups so that a launch still spans the chip.
// ---------------------------------------------------------------------------
template <class Tin, int VEC, int SG>
__global__ void __launch_bounds__(256)
k_colsum(const Tin* __restrict__ part, int64_t p_g, int n_slots, int64_t slot_stride, int64_t ncols, int Jp, int J,
         float* dst, int64_t d_g, int accumulate, float scale, int32_t* nonfinite) {
  constexpr int LANES = 256 / SG;
  __shared__ double red[SG][LANES * VEC];
  const int g = blockIdx.z;
  const int lane = threadIdx.x % LANES, grp = threadIdx.x / LANES;
  const int64_t col0 = ((int64_t)blockIdx.x * LANES + lane) * VEC;
  double s[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) s[e] = 0.0;
  if (col0 < ncols) {
    const Tin* src = part + g * p_g + col0;
    if constexpr (VEC == 4) {
#pragma unroll 4
      for (int q = grp; q < n_slots; q += SG) {
        const float4 v = *(const float4*)(src + (int64_t)q * slot_stride);
        s[0] += (double)v.x;
        s[1] += (double)v.y;
        s[2] += (double)v.z;
        s[3] += (double)v.w;
      }
    } else {
#pragma unroll 8
      for (int q = grp; q < n_slots; q += SG) s[0] += (double)src[(int64_t)q * slot_stride];
    }
  }
#pragma unroll
  for (int e = 0; e < VEC; ++e) red[grp][lane * VEC + e] = s[e];
  __syncthreads();
#pragma unroll
  for (int h = SG / 2; h >= 1; h >>= 1) {
    if (grp < h) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) red[grp][lane * VEC + e] += red[grp + h][lane * VEC + e];
    }
    __syncthreads();
  }
  if (grp == 0 && col0 < ncols) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const int64_t col = col0 + e;
      const double v = red[0][lane * VEC + e];
      const int64_t n = col / Jp;
      const int j = (int)(col % Jp);
      if (j < J) {
        float* o = dst + g * d_g + n * J + j;
        float r = (float)(v * (double)scale);
        if (accumulate) r += *o;
        *o = r;
        if (!__builtin_isfinite(r)) *nonfinite = 1;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// first-layer reverse pass.  Block (s, rc) covers chunk rc of sample s's
// sensor rows and collocation points; per column n it sums
//   q=0   : dA_1 over value rows                       (gs)
//   q=1..3: dA_1 * x_i over value rows                  (gx_i)
//   q=4..6: dA_1 over the d/dx_i rows                   (gd_i; a'_i = W1[:, i])
// into part[g][s][rc][q][n] (fp32; slots beyond d stay zero).
// ---------------------------------------------------------------------------
template <class T>
__global__ void __launch_bounds__(256)
k_first_bwd(FirstBwdArgs<T> p) {
  __shared__ double red[256 * 8];
  const int g = blockIdx.z;
  const int s = blockIdx.x / p.nrc;
  const int rc = blockIdx.x % p.nrc;
  const int W = p.W;
  const int G8 = W / 8;
  const int TPP = G8 < 256 ? G8 : 256;
  const int PPP = 256 / TPP;
  const int lt = threadIdx.x % TPP;
  const int lp = threadIdx.x / TPP;
  const int cg = blockIdx.y * 256 + lt;
  const bool valid = cg < G8;
  const int n0 = cg * 8;
  const int d = p.d;
  double acc[7][8];
#pragma unroll
  for (int q = 0; q < 7; ++q)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[q][e] = 0.0;
  const T* A = p.dA + g * p.a_g;
  if (valid) {
    const int j0 = (int)((int64_t)p.n_s * rc / p.nrc), j1 = (int)((int64_t)p.n_s * (rc + 1) / p.nrc);
    const float* As = p.dAs + g * p.as_g;
    for (int j = j0 + lp; j < j1; j += PPP) {
      float v[8];
      load8<float>(As + ((int64_t)s * p.n_s + j) * p.ldas + n0, v);
      const float* xv = p.xs + g * p.xs_g + (int64_t)j * d;
      double x[3];
#pragma unroll
      for (int i = 0; i < 3; ++i) x[i] = i < d ? (double)xv[i] : 0.0;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        acc[0][e] += (double)v[e];
#pragma unroll
        for (int i = 0; i < 3; ++i) acc[1 + i][e] += (double)v[e] * x[i];
      }
    }
    const int q0 = (int)((int64_t)p.P * rc / p.nrc), q1 = (int)((int64_t)p.P * (rc + 1) / p.nrc);
#pragma unroll 4
    for (int q = q0 + lp; q < q1; q += PPP) {
      const int64_t pt = (int64_t)s * p.P + q;
      float v[8];
      load8<T>(A + pt * p.lda + n0, v);
      const float* xv = p.xc + g * p.xc_g + pt * d;
      float x[3];
#pragma unroll
      for (int i = 0; i < 3; ++i) x[i] = i < d ? xv[i] : 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        acc[0][e] += (double)v[e];
#pragma unroll
        for (int i = 0; i < 3; ++i) acc[1 + i][e] += (double)(v[e] * x[i]);
      }
#pragma unroll
      for (int i = 0; i < 3; ++i) {
        if (i >= p.nd1) continue;
        float u[8];
        load8<T>(A + ((1 + i) * p.n_col + pt) * p.lda + n0, u);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[4 + i][e] += (double)u[e];
      }
    }
  }
  double* out = p.part + (((int64_t)g * p.S + s) * p.nrc + rc) * 7 * W;
#pragma unroll
  for (int q = 0; q < 7; ++q) {
#pragma unroll
    for (int e = 0; e < 8; ++e) red[threadIdx.x * 8 + e] = acc[q][e];
    __syncthreads();
    if (lp == 0 && valid) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        double t = 0.0;
        for (int u = 0; u < PPP; ++u) t += red[(u * TPP + lt) * 8 + e];
        out[(int64_t)q * W + n0 + e] = t;
      }
    }
    __syncthreads();
  }
}

// dW1[n][c] and db1[n] from the partials (fp64 sums, fixed order):
//   c < d : sum_{s,rc} gx_c + gd_c ;  c >= d : sum_{s,rc} gs * z_s[c-d] ;
//   bias (blockIdx.y == in_dim) : sum_{s,rc} gs
__global__ void __launch_bounds__(1024)
k_first_wgrad(const double* __restrict__ part, int S, int nrc, int W, int d, int nd1, int in_dim,
              const float* __restrict__ z, int64_t z_g, int n_z, float* grad, int64_t g_g, int accumulate,
              float scale, int32_t* nonfinite) {
  __shared__ double red[32][32];
  const int g = blockIdx.z;
  const int c = blockIdx.y;
  const int lane = threadIdx.x & 31, grp = threadIdx.x >> 5;   // 32 sample groups
  const int n = blockIdx.x * 32 + lane;
  double acc = 0.0;
  if (n < W) {
    const double* pp = part + (int64_t)g * S * nrc * 7 * W + n;
    const bool xcol = c < d;                       // weight of coordinate c: sum of gx_c and gd_c
    const bool two = xcol && c < nd1;
    const int64_t o1 = xcol ? (int64_t)(1 + c) * W : 0, o2 = (int64_t)(4 + c) * W;
    for (int s = grp; s < S; s += 32) {
      const double* b = pp + (int64_t)s * nrc * 7 * W;
      double t = 0.0;
#pragma unroll 4
      for (int r = 0; r < nrc; ++r) {
        t += b[(int64_t)r * 7 * W + o1];
        if (two) t += b[(int64_t)r * 7 * W + o2];
      }
      if (!xcol && c < in_dim) t *= (double)z[g * z_g + (int64_t)s * n_z + (c - d)];
      acc += t;
    }
  }
  red[grp][lane] = acc;
  __syncthreads();
  if (grp == 0 && n < W) {
    double v = 0.0;
#pragma unroll
    for (int q = 0; q < 32; ++q) v += red[q][lane];
    const int64_t o = c < in_dim ? (int64_t)n * in_dim + c : (int64_t)W * in_dim + n;
    float* dst = grad + g * g_g + o;
    float r = (float)(v * (double)scale);
    if (accumulate) r += *dst;
    *dst = r;
    if (!__builtin_isfinite(r)) *nonfinite = 1;
  }
}

// ---------------------------------------------------------------------------
// losses from the accumulated sums (double): acc[g] = {sum D(fake),
// sum D(real), sum r^2, sum (|grad D| - 1)^2 over the penalty pairs}; the
// penalty P = w lambda_gp acc[3] / n_gp is part of L_D and also stored in gp
// (when gp is not null)
// ---------------------------------------------------------------------------
__global__ void k_losses(const double* __restrict__ acc, int acc_stride, const float* __restrict__ w_group,
                         int S, int B, int64_t SP, float lambda_pde, float lambda_gp, int n_gp, float* loss, float* gp,
                         int32_t* nonfinite, int G) {
  const int g = blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= G) return;
  const double w = w_group ? (double)w_group[g] : 1.0;
  const double* a = acc + g * acc_stride;
  const double Pg = n_gp > 0 ? w * (double)lambda_gp * a[3] / (double)n_gp : 0.0;
  const double LD = w * (a[0] / S - a[1] / B) + Pg;
  const double La = -w * a[0] / S;
  const double Lp = w * (double)lambda_pde * a[2] / (double)SP;
  loss[3 * g + 0] = (float)LD;
  loss[3 * g + 1] = (float)La;
  loss[3 * g + 2] = (float)Lp;
  if (gp) gp[g] = (float)Pg;
  if (!__builtin_isfinite(LD) || !__builtin_isfinite(La) || !__builtin_isfinite(Lp)) *nonfinite = 1;
}

__global__ void k_zero(double* acc, int n, int32_t* flag) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) acc[i] = 0.0;
  if (i == 0 && flag) *flag = 0;
}

// ---------------------------------------------------------------------------
// weight casts: src fp32 [N][K] -> dst [N][Kp] (zero padded) and optionally
// dstT [Kp][N].  With dstT, k_cast_tr goes through 32 x 32 tiles in LDS so
// that both outputs are stored in whole rows (a direct transposed store
// writes one element per row of dstT); k_cast serves dst alone.
// ---------------------------------------------------------------------------
template <class T>
__global__ void __launch_bounds__(256)
k_cast_tr(const float* __restrict__ src, int64_t s_g, int N, int K, int Kp, T* __restrict__ dst,
          T* __restrict__ dstT, int64_t d_g) {
  __shared__ T tile[32][33];
  const int g = blockIdx.z;
  const int k0 = blockIdx.x * 32, n0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
#pragma unroll
  for (int r = ty; r < 32; r += 8) {
    const int n = n0 + r, k = k0 + tx;
    T tv = Elem<T>::from_f(0.0f);
    if (n < N && k < Kp) {
      tv = Elem<T>::from_f(k < K ? src[g * s_g + (int64_t)n * K + k] : 0.0f);
      if (dst) dst[g * d_g + (int64_t)n * Kp + k] = tv;
    }
    tile[r][tx] = tv;
  }
  __syncthreads();
#pragma unroll
  for (int r = ty; r < 32; r += 8) {
    const int k = k0 + r, n = n0 + tx;
    if (k < Kp && n < N) dstT[g * d_g + (int64_t)k * N + n] = tile[tx][r];
  }
}

// split-product weight copies: fp32 src [N][K] -> dst [N][Kp] and dstT
// [Kp][N] with every 16-element block of a row stored as its 16 high bf16
// pieces followed by its 16 low pieces (hi = RNE(w), lo = RNE(w - hi)): the
// rows keep the fp32 byte pitch, and a 64-byte k-slice of a row is exactly
// the split layout the split-product GEMM stages in LDS (padding: zeros)
__device__ __forceinline__ void pair_put(bf16* row, int k, float v) {
  const bf16 hi = (bf16)v;
  const bf16 lo = (bf16)(v - (float)hi);
  row[32 * (k >> 4) + (k & 15)] = hi;
  row[32 * (k >> 4) + 16 + (k & 15)] = lo;
}

__global__ void __launch_bounds__(256)
k_cast_pair(const float* __restrict__ src, int64_t s_g, int N, int K, int Kp, float* __restrict__ dst,
            float* __restrict__ dstT, int64_t d_g) {
  __shared__ float tile[32][33];
  const int g = blockIdx.z;
  const int k0 = blockIdx.x * 32, n0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  bf16* d = dst ? (bf16*)(dst + g * d_g) : nullptr;
  bf16* dT = dstT ? (bf16*)(dstT + g * d_g) : nullptr;
#pragma unroll
  for (int r = ty; r < 32; r += 8) {
    const int n = n0 + r, k = k0 + tx;
    float v = 0.0f;
    if (n < N && k < Kp) {
      v = k < K ? src[g * s_g + (int64_t)n * K + k] : 0.0f;
      if (dst) pair_put(d + (int64_t)n * 2 * Kp, k, v);
    }
    tile[r][tx] = v;
  }
  if (!dstT) return;
  __syncthreads();
#pragma unroll
  for (int r = ty; r < 32; r += 8) {
    const int k = k0 + r, n = n0 + tx;
    if (k < Kp && n < N) pair_put(dT + (int64_t)k * 2 * N, n, tile[tx][r]);
  }
}

// two-term weights: dst[n] = [hi(W[n][:]) | lo(W[n][:])] (2 K wide), with
// hi = W rounded to the storage type and lo = W - hi rounded likewise
template <class T>
__global__ void k_cast2(const float* __restrict__ src, int64_t s_g, int N, int K, T* __restrict__ dst, int64_t d_g) {
  const int g = blockIdx.z;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)N * K) return;
  const int64_t n = idx / K, k = idx % K;
  const float v = src[g * s_g + idx];
  const T hi = Elem<T>::from_f(v);
  const T lo = Elem<T>::from_f(v - Elem<T>::to_f(hi));
  dst[g * d_g + n * 2 * K + k] = hi;
  dst[g * d_g + n * 2 * K + K + k] = lo;
}

template <class T>
__global__ void k_cast(const float* __restrict__ src, int64_t s_g, int N, int K, int Kp, T* __restrict__ dst,
                       T* __restrict__ dstT, int64_t d_g) {
  const int g = blockIdx.z;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)N * Kp) return;
  const int n = (int)(idx / Kp), k = (int)(idx % Kp);
  const float v = k < K ? src[g * s_g + (int64_t)n * K + k] : 0.0f;
  const T tv = Elem<T>::from_f(v);
  if (dst) dst[g * d_g + idx] = tv;
  if (dstT) dstT[g * d_g + (int64_t)k * N + n] = tv;
}

// ===========================================================================
// host launchers
// ===========================================================================
static inline unsigned nblk(int64_t n, int b) { return (unsigned)((n + b - 1) / b); }

hipError_t launch_zproj(const float* p1, int64_t p_g, int in_dim, int d, int W, const float* z, int64_t z_g,
                        int n_z, int S, float* zp, int64_t zp_g, int G, hipStream_t st) {
  k_zproj<<<dim3(nblk((int64_t)S * W, 256), 1, G), 256, 0, st>>>(p1, p_g, in_dim, d, W, z, z_g, n_z, S, zp, zp_g);
  return hipGetLastError();
}

template <class T, bool X64>
static hipError_t first_fwd_nd(int nd1, int nd2, const FirstArgs<T>& a, dim3 grid, hipStream_t st) {
  switch (nd1 * 10 + nd2) {
    case 0: k_first_fwd<T, 0, 0, X64><<<grid, 256, 0, st>>>(a); break;
    case 10: k_first_fwd<T, 1, 0, X64><<<grid, 256, 0, st>>>(a); break;
    case 20: k_first_fwd<T, 2, 0, X64><<<grid, 256, 0, st>>>(a); break;
    case 30: k_first_fwd<T, 3, 0, X64><<<grid, 256, 0, st>>>(a); break;
    case 11: k_first_fwd<T, 1, 1, X64><<<grid, 256, 0, st>>>(a); break;
    case 22: k_first_fwd<T, 2, 2, X64><<<grid, 256, 0, st>>>(a); break;
    case 33: k_first_fwd<T, 3, 3, X64><<<grid, 256, 0, st>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <class T>
hipError_t launch_first_fwd(int nd1, int nd2, const FirstArgs<T>& a, int G, hipStream_t st) {
  if (a.seg.n_points <= 0) return hipSuccess;
  dim3 grid(nblk(a.seg.n_points, FF_PPB), 1, G);
  if constexpr (sizeof(T) == 4) {
    if (a.exact) return first_fwd_nd<T, true>(nd1, nd2, a, grid, st);
  }
  return first_fwd_nd<T, false>(nd1, nd2, a, grid, st);
}

template <class T>
hipError_t launch_out_fwd(const T* H, int64_t h_g, int64_t ldh, int64_t R, int64_t n_value, int W,
                          const float* wout, int64_t w_g, float* y, int64_t y_g, int G, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  k_out_fwd<T><<<dim3(nblk(R, 32), 1, G), 256, 0, st>>>(H, h_g, ldh, R, n_value, W, wout, w_g, y, y_g);
  return hipGetLastError();
}

hipError_t launch_residual(const ResidArgs& a, int G, hipStream_t st) {
  if (a.M <= 0) return hipSuccess;
  k_residual<<<dim3(nblk(a.M, 256), 1, G), 256, 0, st>>>(a);
  return hipGetLastError();
}

int residual_blocks(int64_t M) { return (int)nblk(M, 256); }

hipError_t launch_sum_partials(const double* part, int nb, double* acc, int acc_stride, int slot, int G,
                               hipStream_t st) {
  k_sum_partials<<<G, 256, 0, st>>>(part, nb, acc, acc_stride, slot);
  return hipGetLastError();
}

template <class T>
hipError_t launch_snap_fill(const float* yY, int64_t yY_g, const float* yU, int64_t yU_g, int nY, int nU,
                            int n_fake, const float* real, int64_t real_g, int n_real, int n_in, T* X,
                            int64_t x_g, int ldx, int G, hipStream_t st) {
  const int64_t tot = (int64_t)(n_fake + n_real) * ldx;
  if (tot <= 0) return hipSuccess;
  k_snap_fill<T><<<dim3(nblk(tot, 256), 1, G), 256, 0, st>>>(yY, yY_g, yU, yU_g, nY, nU, nY, nU, 0, n_fake, real,
                                                             real_g, n_real, n_in, X, x_g, ldx);
  return hipGetLastError();
}

template <class T>
hipError_t launch_snap_fill_rows(const float* yY, int64_t yY_g, const float* yU, int64_t yU_g, int nY, int nU,
                                 int ld, int offU, int n_fake, const float* real, int64_t real_g, int n_real, int n_in,
                                 T* X, int64_t x_g, int ldx, int G, hipStream_t st) {
  const int64_t tot = (int64_t)(n_fake + n_real) * ldx;
  if (tot <= 0) return hipSuccess;
  k_snap_fill<T><<<dim3(nblk(tot, 256), 1, G), 256, 0, st>>>(yY, yY_g, yU, yU_g, nY, nU, ld, ld, offU, n_fake, real,
                                                             real_g, n_real, n_in, X, x_g, ldx);
  return hipGetLastError();
}

template <class T>
hipError_t launch_gp_mix(const float* yY, int64_t yY_g, const float* yU, int64_t yU_g, int nY, int nU, int ldY,
                         int ldU, int offU, const float* real, int64_t real_g, const float* eps, int64_t eps_g, int b0,
                         int n, int n_in, T* X, int64_t x_g, int ldx, int G, hipStream_t st) {
  const int64_t tot = (int64_t)n * ldx;
  if (tot <= 0) return hipSuccess;
  k_gp_mix<T><<<dim3(nblk(tot, 256), 1, G), 256, 0, st>>>(yY, yY_g, yU, yU_g, nY, nU, ldY, ldU, offU, real, real_g,
                                                          eps, eps_g, b0, n, n_in, X, x_g, ldx);
  return hipGetLastError();
}

hipError_t launch_fill2(float* seed, int64_t s_g, int n, float v0, float v1, int two, int G, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  k_fill2<<<dim3(nblk(n, 256), 1, G), 256, 0, st>>>(seed, s_g, n, v0, v1, two);
  return hipGetLastError();
}

template <class T>
hipError_t launch_gp_norm(const float* gin, int64_t g_g, int n, int n_in, const float* w_group, float scale,
                          double* part, int64_t p_g, T* X, int64_t x_g, int ldx, int G, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  k_gp_norm<T><<<dim3(n, 1, G), 256, 0, st>>>(gin, g_g, n, n_in, w_group, scale, part, p_g, X, x_g, ldx);
  return hipGetLastError();
}

hipError_t launch_disc_seed(const float* score, int64_t sc_g, int n_fake, int n_real, int S_total, int B_total,
                            const float* w_group, float loss_scale, float* seed, double* acc, int acc_stride,
                            int G, hipStream_t st) {
  k_disc_seed<<<G, 256, 0, st>>>(score, sc_g, n_fake, n_real, S_total, B_total, w_group, loss_scale, seed, acc,
                                 acc_stride);
  return hipGetLastError();
}

int out_bwd_blocks(int64_t n_points, int ppb) { return (int)nblk(n_points, ppb); }

template <class T, bool X64>
static hipError_t out_bwd_nd(int nd1, int nd2, const OutBwdArgs<T>& a, dim3 grid, hipStream_t st) {
  switch (nd1 * 10 + nd2) {
    case 0: k_out_bwd<T, 0, 0, X64><<<grid, 256, 0, st>>>(a); break;
    case 10: k_out_bwd<T, 1, 0, X64><<<grid, 256, 0, st>>>(a); break;
    case 20: k_out_bwd<T, 2, 0, X64><<<grid, 256, 0, st>>>(a); break;
    case 30: k_out_bwd<T, 3, 0, X64><<<grid, 256, 0, st>>>(a); break;
    case 11: k_out_bwd<T, 1, 1, X64><<<grid, 256, 0, st>>>(a); break;
    case 22: k_out_bwd<T, 2, 2, X64><<<grid, 256, 0, st>>>(a); break;
    case 33: k_out_bwd<T, 3, 3, X64><<<grid, 256, 0, st>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <class T>
hipError_t launch_out_bwd(int nd1, int nd2, const OutBwdArgs<T>& a, int G, hipStream_t st) {
  if (a.seg.n_points <= 0) return hipSuccess;
  dim3 grid(nblk(a.seg.n_points, a.ppb), 1, G);
  if constexpr (sizeof(T) == 4) {
    if (a.exact) return out_bwd_nd<T, true>(nd1, nd2, a, grid, st);
  }
  return out_bwd_nd<T, false>(nd1, nd2, a, grid, st);
}

template <class T, bool X64>
static hipError_t out2_bwd_nd(int nd1, int nd2, const Out2BwdArgs<T>& a, dim3 grid, hipStream_t st) {
  switch (nd1 * 10 + nd2) {
    case 0: k_out2_bwd<T, 0, 0, X64><<<grid, 256, 0, st>>>(a); break;
    case 11: k_out2_bwd<T, 1, 1, X64><<<grid, 256, 0, st>>>(a); break;
    case 22: k_out2_bwd<T, 2, 2, X64><<<grid, 256, 0, st>>>(a); break;
    case 33: k_out2_bwd<T, 3, 3, X64><<<grid, 256, 0, st>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <class T>
hipError_t launch_out2_bwd(int nd1, int nd2, const Out2BwdArgs<T>& a, int G, hipStream_t st) {
  if (a.seg.n_points <= 0) return hipSuccess;
  dim3 grid(nblk(a.seg.n_points, a.ppb), 1, G);
  if constexpr (sizeof(T) == 4) {
    if (a.exact) return out2_bwd_nd<T, true>(nd1, nd2, a, grid, st);
  }
  return out2_bwd_nd<T, false>(nd1, nd2, a, grid, st);
}

hipError_t launch_concat_rows(const float* a, int64_t a_g, int na, const float* b, int64_t b_g, int nb, int d,
                              float* out, int64_t o_g, int G, hipStream_t st) {
  const int64_t tot = (int64_t)(na + nb) * d;
  if (tot <= 0) return hipSuccess;
  k_concat_rows<<<dim3(nblk(tot, 256), 1, G), 256, 0, st>>>(a, a_g, na, b, b_g, nb, d, out, o_g);
  return hipGetLastError();
}

template <class T>
hipError_t launch_hier_snap(const HierSnap& h, int n_fake, const float* real, int64_t real_g, int n_real, T* X,
                            int64_t x_g, int ldx, int D, hipStream_t st, const float* eps, int64_t eps_g, int b0) {
  const int64_t tot = (int64_t)(n_fake + n_real) * ldx;
  if (tot <= 0 || D <= 0) return hipSuccess;
  if (eps && n_real != 0) return hipErrorInvalidValue;   // interpolates replace the fake rows only
  k_hier_snap<T><<<dim3(nblk(tot, 256), 1, D), 256, 0, st>>>(h, n_fake, real, real_g, n_real, X, x_g, ldx, eps,
                                                             eps_g, b0);
  return hipGetLastError();
}

hipError_t launch_hier_scatter(const HierSnap& h, const float* dX, int64_t dx_g, int ldx, int n_fake, int D,
                               float* gY, float* gU, float* gN, hipStream_t st) {
  if (n_fake <= 0 || D <= 0) return hipSuccess;
  k_hier_scatter<<<n_fake, HS_NTH, 0, st>>>(h, dX, dx_g, ldx, D, gY, gU, gN);
  return hipGetLastError();
}

hipError_t launch_hier_pde_loss(const double* acc, int slot, float lambda_pde, int64_t SP, float* loss, int D,
                                int32_t* nonfinite, hipStream_t st) {
  if (D <= 0) return hipSuccess;
  k_hier_pde_loss<<<nblk(D, 64), 64, 0, st>>>(acc, slot, lambda_pde, SP, loss, D, nonfinite);
  return hipGetLastError();
}

hipError_t launch_fill_f32(float* p, int64_t n, int64_t p_g, float v, int G, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  k_fill_f32<<<dim3(nblk(n, 256), 1, G), 256, 0, st>>>(p, n, p_g, v);
  return hipGetLastError();
}

template <class Tin>
hipError_t launch_colsum(const Tin* part, int64_t p_g, int n_slots, int64_t slot_stride, int64_t ncols, int Jp, int J,
                         float* dst, int64_t d_g, int accumulate, float scale, int32_t* nonfinite, int G,
                         hipStream_t st) {
  if (ncols <= 0) return hipSuccess;
  // four columns per lane where every slot row and group slab is 16-byte
  // aligned and whole (the workspace is 256-byte aligned)
  int vec = 1;
  if constexpr (sizeof(Tin) == 4) {
    if (ncols % 4 == 0 && slot_stride % 4 == 0 && p_g % 4 == 0 && ((uintptr_t)part & 15) == 0) vec = 4;
  }
  // the fewest slot groups that still give 256 blocks (and no more groups than
  // slots; one group when there are at most two slots)
  const int64_t lanes = (ncols + vec - 1) / vec;
  int sg = n_slots <= 2 ? 1 : 8;
  while (sg >= 8 && sg < 128 && 2 * sg <= n_slots && (lanes + 256 / sg - 1) / (256 / sg) * G < 256) sg *= 4;
  const unsigned nb = (unsigned)((lanes + 256 / sg - 1) / (256 / sg));
#define PIGAN_COLSUM(V, S)                                                                                      \
  k_colsum<Tin, V, S><<<dim3(nb, 1, G), 256, 0, st>>>(part, p_g, n_slots, slot_stride, ncols, Jp, J, dst, d_g, \
                                                      accumulate, scale, nonfinite)
  if constexpr (sizeof(Tin) == 4) {
    if (vec == 4) {
      if (sg == 1) PIGAN_COLSUM(4, 1);
      else if (sg == 8) PIGAN_COLSUM(4, 8);
      else if (sg == 32) PIGAN_COLSUM(4, 32);
      else PIGAN_COLSUM(4, 128);
      return hipGetLastError();
    }
  }
  if (sg == 1) PIGAN_COLSUM(1, 1);
  else if (sg == 8) PIGAN_COLSUM(1, 8);
  else if (sg == 32) PIGAN_COLSUM(1, 32);
  else PIGAN_COLSUM(1, 128);
#undef PIGAN_COLSUM
  return hipGetLastError();
}
template hipError_t launch_colsum<float>(const float*, int64_t, int, int64_t, int64_t, int, int, float*, int64_t, int,
                                         float, int32_t*, int, hipStream_t);
template hipError_t launch_colsum<double>(const double*, int64_t, int, int64_t, int64_t, int, int, float*, int64_t,
                                          int, float, int32_t*, int, hipStream_t);

template <class T>
hipError_t launch_first_bwd(const FirstBwdArgs<T>& a, int G, hipStream_t st) {
  if (a.S <= 0) return hipSuccess;
  dim3 grid(a.S * a.nrc, nblk(a.W / 8, 256), G);
  k_first_bwd<T><<<grid, 256, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_first_wgrad(const double* part, int S, int nrc, int W, int d, int nd1, int in_dim, const float* z,
                              int64_t z_g, int n_z, float* grad, int64_t g_g, int accumulate, float scale,
                              int32_t* nonfinite, int G, hipStream_t st) {
  k_first_wgrad<<<dim3(nblk(W, 32), in_dim + 1, G), 1024, 0, st>>>(part, S, nrc, W, d, nd1, in_dim, z, z_g, n_z,
                                                                   grad, g_g, accumulate, scale, nonfinite);
  return hipGetLastError();
}

hipError_t launch_losses(const double* acc, int acc_stride, const float* w_group, int S, int B, int64_t SP,
                         float lambda_pde, float lambda_gp, int n_gp, float* loss, float* gp, int32_t* nonfinite,
                         int G, hipStream_t st) {
  k_losses<<<nblk(G, 64), 64, 0, st>>>(acc, acc_stride, w_group, S, B, SP, lambda_pde, lambda_gp, n_gp, loss, gp,
                                       nonfinite, G);
  return hipGetLastError();
}

hipError_t launch_zero(double* acc, int n, int32_t* flag, hipStream_t st) {
  k_zero<<<nblk(n > 1 ? n : 1, 256), 256, 0, st>>>(acc, n, flag);
  return hipGetLastError();
}

template <class T>
hipError_t launch_cast(const float* src, int64_t s_g, int N, int K, int Kp, T* dst, T* dstT, int64_t d_g, int G,
                       hipStream_t st) {
  if (dstT)
    k_cast_tr<T><<<dim3((unsigned)((Kp + 31) / 32), (unsigned)((N + 31) / 32), G), 256, 0, st>>>(src, s_g, N, K, Kp,
                                                                                                dst, dstT, d_g);
  else
    k_cast<T><<<dim3(nblk((int64_t)N * Kp, 256), 1, G), 256, 0, st>>>(src, s_g, N, K, Kp, dst, dstT, d_g);
  return hipGetLastError();
}

hipError_t launch_cast_pair(const float* src, int64_t s_g, int N, int K, int Kp, float* dst, float* dstT, int64_t d_g,
                            int G, hipStream_t st) {
  if (Kp % 16 != 0 || (dstT && N % 16 != 0)) return hipErrorInvalidValue;   // whole 16-element blocks per row
  k_cast_pair<<<dim3((unsigned)((Kp + 31) / 32), (unsigned)((N + 31) / 32), G), 256, 0, st>>>(src, s_g, N, K, Kp, dst,
                                                                                            dstT, d_g);
  return hipGetLastError();
}

template <class T>
hipError_t launch_cast2(const float* src, int64_t s_g, int N, int K, T* dst, int64_t d_g, int G, hipStream_t st) {
  k_cast2<T><<<dim3(nblk((int64_t)N * K, 256), 1, G), 256, 0, st>>>(src, s_g, N, K, dst, d_g);
  return hipGetLastError();
}
template hipError_t launch_cast2<bf16>(const float*, int64_t, int, int, bf16*, int64_t, int, hipStream_t);
template hipError_t launch_cast2<f16>(const float*, int64_t, int, int, f16*, int64_t, int, hipStream_t);

#define PIGAN_INST(T)                                                                                         \
  template hipError_t launch_first_fwd<T>(int, int, const FirstArgs<T>&, int, hipStream_t);                  \
  template hipError_t launch_out_fwd<T>(const T*, int64_t, int64_t, int64_t, int64_t, int, const float*,       \
                                        int64_t, float*, int64_t, int, hipStream_t);                          \
  template hipError_t launch_snap_fill<T>(const float*, int64_t, const float*, int64_t, int, int, int,         \
                                          const float*, int64_t, int, int, T*, int64_t, int, int, hipStream_t); \
  template hipError_t launch_out_bwd<T>(int, int, const OutBwdArgs<T>&, int, hipStream_t);                    \
  template hipError_t launch_out2_bwd<T>(int, int, const Out2BwdArgs<T>&, int, hipStream_t);                  \
  template hipError_t launch_hier_snap<T>(const HierSnap&, int, const float*, int64_t, int, T*, int64_t, int, int, \
                                          hipStream_t, const float*, int64_t, int);                              \
  template hipError_t launch_snap_fill_rows<T>(const float*, int64_t, const float*, int64_t, int, int, int, int, \
                                               int, const float*, int64_t, int, int, T*, int64_t, int, int,     \
                                               hipStream_t);                                                    \
  template hipError_t launch_first_bwd<T>(const FirstBwdArgs<T>&, int, hipStream_t);                          \
  template hipError_t launch_gp_mix<T>(const float*, int64_t, const float*, int64_t, int, int, int, int, int,  \
                                       const float*, int64_t, const float*, int64_t, int, int, int, T*, int64_t, \
                                       int, int, hipStream_t);                                                  \
  template hipError_t launch_gp_norm<T>(const float*, int64_t, int, int, const float*, float, double*, int64_t, \
                                        T*, int64_t, int, int, hipStream_t);                                    \
  template hipError_t launch_cast<T>(const float*, int64_t, int, int, int, T*, T*, int64_t, int, hipStream_t);
PIGAN_INST(float)
PIGAN_INST(bf16)
PIGAN_INST(f16)
#undef PIGAN_INST

}  // namespace pigan
