// Internal declarations shared by the HIP kernels and the host orchestration
// of libpigan.so.  gfx950 (CDNA4) only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "pigan.h"

namespace pigan {

typedef __bf16 bf16;
typedef _Float16 f16;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// ---------------------------------------------------------------------------
// Element traits.  A matrix-core "chunk" covers 16 values of the contraction
// index: every lane holds 8 consecutive values of its row (16 bytes in bf16 /
// fp16, 32 bytes in fp32).  The same (lane, element) -> k assignment is used
// for both operands, so any k order inside a chunk is consistent.
// ---------------------------------------------------------------------------
template <class T> struct Elem;

template <> struct Elem<float> {
  typedef f32x8 frag;
  static __device__ __forceinline__ float to_f(float v) { return v; }
  static __device__ __forceinline__ float from_f(float v) { return v; }
  static __device__ __forceinline__ void mma(f32x16& acc, const frag& a, const frag& b) {
#pragma unroll
    for (int q = 0; q < 8; ++q) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[q], b[q], acc, 0, 0, 0);
  }
};

template <> struct Elem<bf16> {
  typedef bf16x8 frag;
  static __device__ __forceinline__ float to_f(bf16 v) { return (float)v; }
  static __device__ __forceinline__ bf16 from_f(float v) { return (bf16)v; }
  static __device__ __forceinline__ void mma(f32x16& acc, const frag& a, const frag& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
  }
};

template <> struct Elem<f16> {
  typedef f16x8 frag;
  static __device__ __forceinline__ float to_f(f16 v) { return (float)v; }
  static __device__ __forceinline__ f16 from_f(float v) { return (f16)v; }
  static __device__ __forceinline__ void mma(f32x16& acc, const frag& a, const frag& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc, 0, 0, 0);
  }
};

// ---------------------------------------------------------------------------
// Split products for fp32 storage.  A fragment of 8 fp32 values is cut into
// bf16 pieces x = x0 + x1 (+ x2) by repeated round-to-nearest: each residual
// is exact in fp32, so two pieces carry about 16 significand bits and three
// pieces carry all 24 of an fp32 value.  Products of bf16 pieces are exact in
// the matrix core's fp32 accumulator.
//   PM_SPLIT2: x0 y0 + x0 y1 + x1 y0  (about 2^-16 relative; x1 y1 dropped)
//   PM_SPLIT3: all pieces with i + j <= 2 (the terms dropped are below 2^-24
//              relative), accumulated per operand stage and then in fp64
//              by the kernels, so that long contractions do not round at
//              fp32 precision at every step.
// ---------------------------------------------------------------------------
//   PM_F64:    the fp32 operands go through the fp64 matrix core (exact
//              products, fp64 accumulation), rounded once at the end.
enum ProdMode { PM_NATIVE = 0, PM_SPLIT2 = 2, PM_SPLIT3 = 3, PM_F64 = 4 };
typedef double f64x4 __attribute__((ext_vector_type(4)));

template <int NP>
__device__ __forceinline__ void split_frag(const f32x8& x, bf16x8 (&p)[NP]) {
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    float r = x[q];
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const bf16 h = (bf16)r;
      p[i][q] = h;
      r -= (float)h;
    }
  }
}

// acc += b . a over one 16-wide chunk from split operands (smallest terms first)
template <int NP>
__device__ __forceinline__ void mma_split(f32x16& acc, const bf16x8 (&b)[NP], const bf16x8 (&a)[NP]) {
  if constexpr (NP == 3) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[2], a[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[1], a[1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[0], a[2], acc, 0, 0, 0);
  }
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[1], a[0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[0], a[1], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[0], a[0], acc, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// tanh and its derivatives with respect to the pre-activation a:
//   t = tanh(a), s = dt/da = 1 - t^2, s' = -2 t s, s'' = 2 s (3 t^2 - 1).
// With e = exp(-2|a|):  |t| = (1 - e) / (1 + e),  s = 4 e / (1 + e)^2.
// s is formed from e directly, so it keeps full relative accuracy for
// saturated units where 1 - t^2 would cancel.  e comes from the hardware
// base-2 exponential (about 1e-6 relative for |a| <= 10, the rounding of the
// scaled argument included).  For |a| < 1/8, where 1 - e would cancel, t is
// the odd Taylor series a - a^3/3 + 2a^5/15 - 17a^7/315 + 62a^9/2835
// (truncation below 2e-10 relative there).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void tanh_ts(float a, float& t, float& s) {
  const float ax = fabsf(a);
  const float e = __builtin_amdgcn_exp2f(ax * -2.8853900817779268f);   // -2 / ln 2
  const float r = __builtin_amdgcn_rcpf(1.0f + e);
  const float a2 = a * a;
  float q = 62.0f / 2835.0f;
  q = q * a2 - 17.0f / 315.0f;
  q = q * a2 + 2.0f / 15.0f;
  q = q * a2 - 1.0f / 3.0f;
  float small = a + (a * a2) * q;
  float big = copysignf((1.0f - e) * r, a);
  // both branches are evaluated (a few FMAs) and selected per lane: left as a
  // conditional, the compiler forms divergent branches around each element,
  // which serialises the epilogues' independent tanh evaluations
  asm("" : "+v"(small), "+v"(big));
  t = ax < 0.125f ? small : big;
  s = (4.0f * e) * (r * r);
}

// The same quantities evaluated in fp64 and rounded once (fp32-mode kernels:
// every stored value then carries a single rounding).
__device__ __forceinline__ void tanh_ts64(float a, float& t, float& s) {
  const double x = -2.0 * fabs((double)a);
  const double e = exp(x);
  const double m = expm1(x);
  t = (float)copysign(-m / (2.0 + m), (double)a);
  s = (float)(4.0 * e / ((1.0 + e) * (1.0 + e)));
}

template <bool X64>
__device__ __forceinline__ void tanh_pair(float a, float& t, float& s) {
  if constexpr (X64) tanh_ts64(a, t, s);
  else tanh_ts(a, t, s);
}

// ---------------------------------------------------------------------------
// Launch descriptors (host side builds them, kernels read them by value).
// Row layout of one network's activations for a chunk of samples:
//   rows [0, n_sen)                       sensor points (value stream only)
//   rows [n_sen + k*n_col, n_sen+(k+1)*n_col)  collocation stream k
// with stream order value, d/dx_1..d/dx_d, d^2/dx_1^2..d^2/dx_d^2.  The value
// rows are therefore contiguous: [0, n_sen + n_col).
// ---------------------------------------------------------------------------
struct Seg {
  int64_t n_points;   // points in the segment
  int64_t row0;       // row of stream 0, point 0
  int64_t plane;      // row distance between streams of one point
};

enum EpiMode { EPI_FWD = 0, EPI_BWD = 1, EPI_DF = 2 };

template <class T> struct NtArgs {
  const T* X;  int64_t x_g;  int64_t ldx;  // A operand rows (activations)
  const T* Wm; int64_t w_g;  int64_t ldw;  // B operand rows: [N x K] row-major
  const float* bias; int64_t b_g;         // EPI_FWD: bias on stream 0 (may be null)
  T* out_a;  T* out_h; int64_t o_g; int64_t ldo;  // EPI_FWD: pre-activation / activation
  const T* aprev;                          // EPI_BWD: saved pre-activation of the layer below
  T* out_da;                               // EPI_BWD: its pre-activation cotangent
  float* seedY; float* seedU; int64_t sY_g; int64_t sU_g;  // EPI_DF outputs
  int32_t nY; int32_t nU; float df_sign;
  // EPI_FWD of the last hidden layer with the output layer fused (only where
  // nt_resident_ok holds): y[row] = w_out . h (+ b_out on the value stream),
  // rows in the activation row layout; wout = [w_out (N), b_out]
  float* y; int64_t y_g; const float* wout; int64_t wo_g;
  // second-layer calls with the first layer formed in the kernel (only where
  // nt_resident_ok holds; fp1 != null): the forward builds its operand X,
  // and the reverse pass its saved pre-activations, from the coordinates, the
  // per-sample z-projection (+ b1) and the fp32 W1 instead of reading them.
  // Point pt of the segment is sample pt / fPn at coordinate row
  // (fx_shared ? pt % fPn : pt).
  const float* fp1; int64_t fp_g; int32_t f_in; int32_t f_d;
  const float* fzp; int64_t fzp_g;
  const float* fx; int64_t fx_g; int32_t fx_shared; int64_t fPn;
  T* f_out_h;                              // forward: also store the generated activations (may be null)
  // residual blocks of a shared trunk (tiled kernels only).  EPI_FWD: skip
  // (the activations of layer l - 2, every stream) is added to the
  // activations.  EPI_BWD: skip_g (the total activation cotangent carried
  // back by a skip) is added to the product, and out_gh, when set, receives
  // that total before the reverse carry; out_gh may alias skip_g (a block
  // reads its whole tile of skip_g before the barrier that precedes its
  // stores, and tiles are disjoint).
  const T* skip; const T* skip_g; T* out_gh;
  // EPI_DF: seeds per point are sY_ld / sU_ld apart (0: nY / nU) and the u
  // seeds start sU_off entries into a point's row
  int32_t sY_ld; int32_t sU_ld; int32_t sU_off;
  Seg seg;
  int32_t N, K;
  // fp32 storage: how the products are formed (ProdMode)
  int32_t pm;
  // two-term weights (16-bit storage): K = 2 kx, the weight rows hold
  // [W_hi | W_lo] and the operand X (kx wide) is read twice
  int32_t kx;
};

// per-kernel-family profiling hooks (host)
void prof_begin(hipStream_t st, const char* name, double flops, double bytes);
void prof_end(hipStream_t st);

// ---------------------------------------------------------------------------
// Host launchers (defined in the .hip files)
// ---------------------------------------------------------------------------
template <class T>
hipError_t launch_gemm_nt(int epi, int nd1, int nd2, const NtArgs<T>& a, int G, hipStream_t st);

// pm: ProdMode for fp32 storage; PM_SPLIT3 and PM_F64 write their split
// partials in fp64 to partial64 instead of partial
template <class T>
hipError_t launch_gemm_dw(const T* dA, int64_t a_g, int64_t lda, const T* H, int64_t h_g, int64_t ldh,
                          int64_t R, int64_t n_value, int N, int J, float* partial, double* pdb,
                          int n_split, int64_t rows_per_split, int G, hipStream_t st, int pm = PM_NATIVE,
                          double* partial64 = nullptr);

// whether launch_gemm_nt runs this shape on the persistent resident-weight
// kernel, which alone fuses the output layer and the first layer (16-bit
// storage, K = N = 128, at most 5 streams, rows addressable with 32-bit
// offsets)
bool nt_resident_ok(int elem_bytes, int C, int K, int N, int64_t n_points, int64_t ldx, int64_t ldo);

void dw_split_plan(int64_t R, int N, int J, int elem_bytes, int G, int* n_split, int64_t* rows_per_split);

}  // namespace pigan
