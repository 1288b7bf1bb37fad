// Matrix-core (MFMA) kernels of the PI-GAN step for gfx950.
//
// k_gemm_nt  : C_k = X_k . W^T for the C jet streams of a tile of points,
//              with three fused epilogues:
//   EPI_FWD  hidden-layer forward: adds the bias to the value stream, applies
//            tanh and carries the spatial derivatives forward
//              h = t, h'_i = s a'_i, h''_i = s a''_i + s' (a'_i)^2
//            (chain rule of the generator's induced derivative network,
//            Sec. III.B.1); writes the pre-activations (kept for the reverse
//            pass) and the activations.
//   EPI_BWD  reverse pass: the product is dH of the layer below; the epilogue
//            turns it into that layer's pre-activation cotangents
//              g_a   = s g_h + sum_i s' a'_i g_h'_i + (s' a''_i + s'' a'_i^2) g_h''_i
//              g_a'_i = s g_h'_i + 2 s' a'_i g_h''_i,   g_a''_i = s g_h''_i
//   EPI_DF   reverse pass through the discriminator's first layer for the
//            fake snapshots: writes -dL_D/dF into the generators' sensor-row
//            cotangents (the adversarial generator loss is the negated
//            critic term).
// k_gemm_dw  : dW = sum_rows dA^T H (split over rows, fp32 partials), plus
//              the bias cotangent sum over the value rows.
// The split partials are summed in fp64, in split order, by k_colsum.
//
// Tiles: a 64-lane wave owns 32 points x 32*NT columns for every stream; the
// block is WM x WN waves.  Operands are staged through LDS in 64-byte k-slices
// (80-byte row pitch, conflict-free 16-byte fragment reads) with the next
// slice prefetched into registers while the current one is multiplied.
#include "common.h"

namespace pigan {

static constexpr int LDS_PITCH = 80;

template <class T, int ND1, int ND2, int WM, int WN, int NT, int EPI>
__global__ void __launch_bounds__(64 * WM * WN)
k_gemm_nt(const NtArgs<T> p) {
  constexpr int C = 1 + ND1 + ND2;
  constexpr int BM = 32 * WM;
  constexpr int BN = 32 * NT * WN;
  constexpr int NTH = 64 * WM * WN;
  constexpr int KS = 64 / (int)sizeof(T);          // k values per stage
  constexpr int NCH = 64 / (16 * (int)sizeof(T));  // 16-wide chunks per stage
  constexpr int ROWS = C * BM + BN;
  constexpr int PIECES = ROWS * 4;
  constexpr int PPT = (PIECES + NTH - 1) / NTH;
  typedef typename Elem<T>::frag frag;
  __shared__ __attribute__((aligned(16))) char lds[ROWS * LDS_PITCH];

  const int g = blockIdx.z;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % WM;
  const int wn = wave / WM;
  const int64_t m0 = (int64_t)blockIdx.x * BM;
  const int n0 = blockIdx.y * BN;
  const int64_t npts = p.seg.n_points;

  const char* Xb = (const char*)(p.X + g * p.x_g);
  const char* Wb = (const char*)(p.Wm + g * p.w_g);

  int64_t srcoff[PPT];
  bool valid[PPT];
#pragma unroll
  for (int i = 0; i < PPT; ++i) {
    const int piece = tid + i * NTH;
    const int row = piece >> 2, sg = piece & 3;
    valid[i] = false;
    srcoff[i] = 0;
    if (piece < PIECES) {
      if (row < C * BM) {
        const int k = row / BM, pp = row % BM;
        const int64_t pt = m0 + pp;
        valid[i] = pt < npts;
        srcoff[i] = (p.seg.row0 + k * p.seg.plane + pt) * p.ldx * (int64_t)sizeof(T) + sg * 16;
      } else {
        const int n = n0 + row - C * BM;
        valid[i] = n < p.N;
        srcoff[i] = (int64_t)n * p.ldw * (int64_t)sizeof(T) + sg * 16;
      }
    }
  }

  f32x16 acc[C][NT];
#pragma unroll
  for (int k = 0; k < C; ++k)
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[k][t][r] = 0.0f;

  uint4 buf[PPT];
  auto gload = [&](int kt) {
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int piece = tid + i * NTH;
      const int row = piece >> 2;
      if (valid[i]) {
        const char* base = row < C * BM ? Xb : Wb;
        buf[i] = *(const uint4*)(base + srcoff[i] + (int64_t)kt * 64);
      } else {
        buf[i] = make_uint4(0u, 0u, 0u, 0u);
      }
    }
  };

  const int nk = p.K / KS;
  gload(0);
  for (int kt = 0; kt < nk; ++kt) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int piece = tid + i * NTH;
      if (piece < PIECES) *(uint4*)(lds + (piece >> 2) * LDS_PITCH + (piece & 3) * 16) = buf[i];
    }
    __syncthreads();
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int koff = c * 32 + (lane >> 5) * (8 * (int)sizeof(T));
      frag bfr[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t)
        bfr[t] = *(const frag*)(lds + (C * BM + 32 * (wn * NT + t) + (lane & 31)) * LDS_PITCH + koff);
#pragma unroll
      for (int k = 0; k < C; ++k) {
        const frag afr = *(const frag*)(lds + (k * BM + 32 * wm + (lane & 31)) * LDS_PITCH + koff);
#pragma unroll
        for (int t = 0; t < NT; ++t) Elem<T>::mma(acc[k][t], afr, bfr[t]);
      }
    }
  }

  // ---- epilogue: lane owns column (lane & 31) and 16 rows of every 32x32 tile
  const int hh = lane >> 5;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int n = n0 + 32 * (wn * NT + t) + (lane & 31);
    if (n >= p.N) continue;
    float bn = 0.0f;
    if (EPI == EPI_FWD && p.bias) bn = p.bias[g * p.b_g + n];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t pt = m0 + 32 * wm + 8 * (r >> 2) + 4 * hh + (r & 3);
      if (pt >= npts) continue;
      int64_t o[C];
#pragma unroll
      for (int k = 0; k < C; ++k) o[k] = g * p.o_g + (p.seg.row0 + k * p.seg.plane + pt) * p.ldo + n;
      if (EPI == EPI_FWD) {
        const float a0 = acc[0][t][r] + bn;
        float tt, s;
        tanh_ts(a0, tt, s);
        const float sp = -2.0f * tt * s;
        if (p.out_a) {
          p.out_a[o[0]] = Elem<T>::from_f(a0);
#pragma unroll
          for (int k = 1; k < C; ++k) p.out_a[o[k]] = Elem<T>::from_f(acc[k][t][r]);
        }
        p.out_h[o[0]] = Elem<T>::from_f(tt);
#pragma unroll
        for (int i = 0; i < ND1; ++i) p.out_h[o[1 + i]] = Elem<T>::from_f(s * acc[1 + i][t][r]);
#pragma unroll
        for (int i = 0; i < ND2; ++i) {
          const float a1 = acc[1 + i][t][r];
          p.out_h[o[1 + ND1 + i]] = Elem<T>::from_f(s * acc[1 + ND1 + i][t][r] + sp * a1 * a1);
        }
      } else if (EPI == EPI_BWD) {
        float ap[C];
#pragma unroll
        for (int k = 0; k < C; ++k) ap[k] = Elem<T>::to_f(p.aprev[o[k]]);
        float tt, s;
        tanh_ts(ap[0], tt, s);
        const float sp = -2.0f * tt * s;
        const float spp = 2.0f * s * (3.0f * tt * tt - 1.0f);
        float ga = s * acc[0][t][r];
#pragma unroll
        for (int i = 0; i < ND1; ++i) ga += sp * ap[1 + i] * acc[1 + i][t][r];
#pragma unroll
        for (int i = 0; i < ND2; ++i)
          ga += (sp * ap[1 + ND1 + i] + spp * ap[1 + i] * ap[1 + i]) * acc[1 + ND1 + i][t][r];
        p.out_da[o[0]] = Elem<T>::from_f(ga);
#pragma unroll
        for (int i = 0; i < ND1; ++i) {
          float gd = s * acc[1 + i][t][r];
          if (i < ND2) gd += 2.0f * sp * ap[1 + i] * acc[1 + ND1 + i][t][r];
          p.out_da[o[1 + i]] = Elem<T>::from_f(gd);
        }
#pragma unroll
        for (int i = 0; i < ND2; ++i) p.out_da[o[1 + ND1 + i]] = Elem<T>::from_f(s * acc[1 + ND1 + i][t][r]);
      } else {  // EPI_DF: rows are fake snapshots (samples), columns snapshot entries
        const float v = p.df_sign * acc[0][t][r];
        if (n < p.nY) p.seedY[g * p.sY_g + pt * p.nY + n] = v;
        else if (n < p.nY + p.nU) p.seedU[g * p.sU_g + pt * p.nU + (n - p.nY)] = v;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// dW[n][j] = sum_{rows m} dA[m][n] H[m][j]   (contraction over rows)
// Each block owns a (BNn x BJ) output tile and one contiguous range of rows.
// Row slices are transposed into LDS ([column][row], 80-byte pitch) so that
// the fragments (8 consecutive rows of one column) are 16-byte reads.
// ---------------------------------------------------------------------------
template <class T, int WM, int WN, int NT>
__global__ void __launch_bounds__(64 * WM * WN)
k_gemm_dw(const T* __restrict__ dA, int64_t a_g, int64_t lda, const T* __restrict__ H, int64_t h_g,
          int64_t ldh, int64_t R, int64_t n_value, int N, int J, float* __restrict__ partial,
          double* __restrict__ pdb, int n_split, int64_t rows_per_split) {
  constexpr int BNn = 32 * NT * WM;
  constexpr int BJ = 32 * NT * WN;
  constexpr int NTH = 64 * WM * WN;
  constexpr int ES = (int)sizeof(T);
  constexpr int SR = 64 / ES;               // rows per stage
  constexpr int EPP = 16 / ES;              // elements per 16-byte load
  constexpr int RPP = ES == 2 ? 2 : 1;      // rows per piece (packed LDS writes)
  constexpr int NCH = 64 / (16 * ES);
  constexpr int PA = (SR / RPP) * (BNn / EPP);
  constexpr int PB = (SR / RPP) * (BJ / EPP);
  constexpr int PIECES = PA + PB;
  constexpr int PPT = (PIECES + NTH - 1) / NTH;
  typedef typename Elem<T>::frag frag;
  __shared__ __attribute__((aligned(16))) char lds[(BNn + BJ) * LDS_PITCH];

  const int tiles_n = (N + BNn - 1) / BNn;
  const int tn = blockIdx.x % tiles_n;
  const int tj = blockIdx.x / tiles_n;
  const int split = blockIdx.y;
  const int g = blockIdx.z;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % WM;
  const int wn = wave / WM;
  const int n0 = tn * BNn;
  const int j0 = tj * BJ;
  const int64_t r0 = (int64_t)split * rows_per_split;
  const int64_t r1 = r0 + rows_per_split < R ? r0 + rows_per_split : R;
  const int64_t rv = r1 < n_value ? r1 : n_value;

  const T* A = dA + g * a_g;
  const T* B = H + g * h_g;

  f32x16 acc[NT][NT];
#pragma unroll
  for (int a = 0; a < NT; ++a)
#pragma unroll
    for (int b = 0; b < NT; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;
  double dbacc = 0.0;

  uint4 buf[PPT][RPP];
  auto gload = [&](int64_t k0) {
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int piece = tid + i * NTH;
      const bool isA = piece < PA;
      const int q = isA ? piece : piece - PA;
      const int ncg = (isA ? BNn : BJ) / EPP;
      const int rp = q / ncg, cg = q % ncg;
      const int col = (isA ? n0 : j0) + cg * EPP;
      const int lim = isA ? N : J;
#pragma unroll
      for (int u = 0; u < RPP; ++u) {
        const int64_t row = k0 + rp * RPP + u;
        if (piece < PIECES && row < r1 && col < lim) {
          buf[i][u] = isA ? *(const uint4*)(A + row * lda + col) : *(const uint4*)(B + row * ldh + col);
        } else {
          buf[i][u] = make_uint4(0u, 0u, 0u, 0u);
        }
      }
    }
  };

  gload(r0);
  for (int64_t k0 = r0; k0 < r1; k0 += SR) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int piece = tid + i * NTH;
      if (piece >= PIECES) continue;
      const bool isA = piece < PA;
      const int q = isA ? piece : piece - PA;
      const int ncg = (isA ? BNn : BJ) / EPP;
      const int rp = q / ncg, cg = q % ncg;
      char* base = lds + (isA ? 0 : BNn * LDS_PITCH);
      if (ES == 2) {
        const uint16_t* lo = (const uint16_t*)&buf[i][0];
        const uint16_t* hi = (const uint16_t*)&buf[i][RPP - 1];
#pragma unroll
        for (int e = 0; e < EPP; ++e) {
          const uint32_t w = (uint32_t)lo[e] | ((uint32_t)hi[e] << 16);
          *(uint32_t*)(base + (cg * EPP + e) * LDS_PITCH + rp * 4) = w;
        }
      } else {
        const uint32_t* v = (const uint32_t*)&buf[i][0];
#pragma unroll
        for (int e = 0; e < EPP; ++e) *(uint32_t*)(base + (cg * EPP + e) * LDS_PITCH + rp * 4) = v[e];
      }
    }
    __syncthreads();
    if (k0 + SR < r1) gload(k0 + SR);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int koff = c * 32 + (lane >> 5) * (8 * ES);
      frag af[NT], bf[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        af[t] = *(const frag*)(lds + (32 * (wm * NT + t) + (lane & 31)) * LDS_PITCH + koff);
        bf[t] = *(const frag*)(lds + (BNn + 32 * (wn * NT + t) + (lane & 31)) * LDS_PITCH + koff);
      }
#pragma unroll
      for (int a = 0; a < NT; ++a)
#pragma unroll
        for (int b = 0; b < NT; ++b) Elem<T>::mma(acc[a][b], af[a], bf[b]);
    }
    // bias cotangent: value rows of this slice, one column per thread
    if (pdb && tj == 0 && tid < BNn && k0 < rv) {
      const int nr = (int)((rv - k0) < SR ? (rv - k0) : SR);
      const T* colp = (const T*)(lds + tid * LDS_PITCH);
      float part_sum = 0.0f;
      for (int u = 0; u < nr; ++u) part_sum += Elem<T>::to_f(colp[u]);
      dbacc += (double)part_sum;
    }
  }

  const int hh = lane >> 5;
  float* out = partial + ((int64_t)g * n_split + split) * (int64_t)N * J;
#pragma unroll
  for (int a = 0; a < NT; ++a) {
#pragma unroll
    for (int b = 0; b < NT; ++b) {
      const int j = j0 + 32 * (wn * NT + b) + (lane & 31);
      if (j >= J) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int n = n0 + 32 * (wm * NT + a) + 8 * (r >> 2) + 4 * hh + (r & 3);
        if (n < N) out[(int64_t)n * J + j] = acc[a][b][r];
      }
    }
  }
  if (pdb && tj == 0 && tid < BNn && n0 + tid < N)
    pdb[((int64_t)g * n_split + split) * N + n0 + tid] = dbacc;
}

// ---------------------------------------------------------------------------
// host launchers
// ---------------------------------------------------------------------------
namespace {

template <class T, int ND1, int ND2, int EPI>
hipError_t nt_dispatch_tile(const NtArgs<T>& a, int G, hipStream_t st) {
  constexpr int C = 1 + ND1 + ND2;
  const int64_t npts = a.seg.n_points;
  if (npts <= 0) return hipSuccess;
  if (a.N <= 32) {
    dim3 grid((unsigned)((npts + 127) / 128), (unsigned)((a.N + 31) / 32), G);
    k_gemm_nt<T, ND1, ND2, 4, 1, 1, EPI><<<grid, 256, 0, st>>>(a);
  } else if (a.N <= 64 || C > 5) {
    dim3 grid((unsigned)((npts + 63) / 64), (unsigned)((a.N + 63) / 64), G);
    k_gemm_nt<T, ND1, ND2, 2, 2, 1, EPI><<<grid, 256, 0, st>>>(a);
  } else {
    dim3 grid((unsigned)((npts + 63) / 64), (unsigned)((a.N + 127) / 128), G);
    k_gemm_nt<T, ND1, ND2, 2, 2, 2, EPI><<<grid, 256, 0, st>>>(a);
  }
  return hipGetLastError();
}

template <class T, int EPI>
hipError_t nt_dispatch_streams(int nd1, int nd2, const NtArgs<T>& a, int G, hipStream_t st) {
  const int key = nd1 * 10 + nd2;
  switch (key) {
    case 0: return nt_dispatch_tile<T, 0, 0, EPI>(a, G, st);
    case 10: return nt_dispatch_tile<T, 1, 0, EPI>(a, G, st);
    case 20: return nt_dispatch_tile<T, 2, 0, EPI>(a, G, st);
    case 30: return nt_dispatch_tile<T, 3, 0, EPI>(a, G, st);
    case 11: return nt_dispatch_tile<T, 1, 1, EPI>(a, G, st);
    case 22: return nt_dispatch_tile<T, 2, 2, EPI>(a, G, st);
    case 33: return nt_dispatch_tile<T, 3, 3, EPI>(a, G, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

template <class T>
hipError_t launch_gemm_nt(int epi, int nd1, int nd2, const NtArgs<T>& a, int G, hipStream_t st) {
  if (epi == EPI_FWD) return nt_dispatch_streams<T, EPI_FWD>(nd1, nd2, a, G, st);
  if (epi == EPI_BWD) return nt_dispatch_streams<T, EPI_BWD>(nd1, nd2, a, G, st);
  if (nd1 != 0 || nd2 != 0) return hipErrorInvalidValue;
  return nt_dispatch_tile<T, 0, 0, EPI_DF>(a, G, st);
}

void dw_split_plan(int64_t R, int N, int J, int elem_bytes, int G, int* n_split, int64_t* rows_per_split) {
  const int SR = 64 / elem_bytes;
  const int bt = (N >= 128 && J >= 128) ? 128 : ((N >= 64 && J >= 64) ? 64 : 32);
  const int64_t tiles = (int64_t)((N + bt - 1) / bt) * ((J + bt - 1) / bt) * G;
  int64_t want = (1024 + tiles - 1) / tiles;
  const int64_t stages = (R + SR - 1) / SR;
  int64_t max_split = stages / 4 > 0 ? stages / 4 : 1;
  if (want > max_split) want = max_split;
  if (want < 1) want = 1;
  if (want > 65535) want = 65535;
  int64_t rps = (R + want - 1) / want;
  rps = (rps + SR - 1) / SR * SR;
  if (rps <= 0) rps = SR;
  *rows_per_split = rps;
  *n_split = (int)((R + rps - 1) / rps);
  if (*n_split < 1) *n_split = 1;
}

template <class T>
hipError_t launch_gemm_dw(const T* dA, int64_t a_g, int64_t lda, const T* H, int64_t h_g, int64_t ldh,
                          int64_t R, int64_t n_value, int N, int J, float* partial, double* pdb,
                          int n_split, int64_t rows_per_split, int G, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  if (N >= 128 && J >= 128) {
    dim3 grid((unsigned)(((N + 127) / 128) * ((J + 127) / 128)), n_split, G);
    k_gemm_dw<T, 2, 2, 2><<<grid, 256, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, J, partial, pdb,
                                                 n_split, rows_per_split);
  } else if (N >= 64 && J >= 64) {
    dim3 grid((unsigned)(((N + 63) / 64) * ((J + 63) / 64)), n_split, G);
    k_gemm_dw<T, 2, 2, 1><<<grid, 256, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, J, partial, pdb,
                                                 n_split, rows_per_split);
  } else {
    dim3 grid((unsigned)(((N + 31) / 32) * ((J + 31) / 32)), n_split, G);
    k_gemm_dw<T, 1, 1, 1><<<grid, 64, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, J, partial, pdb,
                                                n_split, rows_per_split);
  }
  return hipGetLastError();
}

#define PIGAN_INST(T)                                                                                    \
  template hipError_t launch_gemm_nt<T>(int, int, int, const NtArgs<T>&, int, hipStream_t);              \
  template hipError_t launch_gemm_dw<T>(const T*, int64_t, int64_t, const T*, int64_t, int64_t, int64_t, \
                                        int64_t, int, int, float*, double*, int, int64_t, int, hipStream_t);
PIGAN_INST(float)
PIGAN_INST(bf16)
PIGAN_INST(f16)
#undef PIGAN_INST

}  // namespace pigan
