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
//            fake snapshots: writes -dL_D/dF (the adversarial generator loss
//            is the negated critic term) into the generators' sensor-row
//            cotangents, or into a per-critic input-cotangent array.
//   Residual blocks of a shared trunk add the skip activations (forward) and
//   the skip cotangent (reverse) in the same epilogues.
// k_gemm_dw  : dW = sum_rows dA^T H (split over rows, fp32 partials), plus
//              the bias cotangent sum over the value rows.
// The split partials are summed in fp64, in a fixed order, by k_colsum.
//
// Tiles: a 64-lane wave owns 32 points x 32*NT columns for every stream; the
// block is WM x WN waves.  The MFMA computes W . X^T so that a lane holds one
// point and runs of four columns (vector stores, lane-local derivative
// carry).  Operands are staged through LDS in 64-byte k-slices (swizzled
// segments, conflict-free writes and fragment reads): wide layers load them
// straight into a 3- or 4-deep LDS ring, the others prefetch the next slices
// into registers while the current one is multiplied.
#include "common.h"

namespace pigan {

// Operand stages of k_gemm_nt: 64-byte rows (one k-slice) with the four
// 16-byte segments of row r stored in the order s ^ ((r >> 2) & 3).  The
// fragment reads (32 consecutive rows, one segment) and the stage writes (four
// lanes per row) are then both free of bank conflicts (measured with the
// LDS bank-conflict counter; a padded pitch without the swizzle conflicted on
// the writes).
static constexpr int LDS_PITCH = 64;
typedef uint32_t u32x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ int lds_seg(int row, int seg) { return row * LDS_PITCH + ((seg ^ ((row >> 2) & 3)) << 4); }

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own
// L2).  Map hardware block b to a logical tile so that every XCD walks one
// contiguous range of logical tiles: blocks that share an operand tile run on
// the same XCD at about the same time.  Bijective for any block count.
__device__ __forceinline__ int64_t xcd_remap(int64_t b, int64_t nb) {
  const int64_t q = nb / 8, r = nb % 8;
  const int64_t x = b % 8, local = b / 8;
  return x < r ? x * (q + 1) + local : r * (q + 1) + (x - r) * q + local;
}

// four consecutive elements in the storage type (8 bytes in bf16/fp16, 16 in fp32)
template <class T>
__device__ __forceinline__ void store4(T* p, const float* v) {
  if (sizeof(T) == 2) {
    uint2 raw;
    T* e = (T*)&raw;
#pragma unroll
    for (int i = 0; i < 4; ++i) e[i] = Elem<T>::from_f(v[i]);
    *(uint2*)p = raw;
  } else {
    *(float4*)p = make_float4(v[0], v[1], v[2], v[3]);
  }
}

template <class T>
__device__ __forceinline__ void load4(const T* p, float* v) {
  if (sizeof(T) == 2) {
    const uint2 raw = *(const uint2*)p;
    const T* e = (const T*)&raw;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = Elem<T>::to_f(e[i]);
  } else {
    const float4 a = *(const float4*)p;
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  }
}

// Barrier for data exchanged through LDS only.  __syncthreads() also fences
// global memory, which makes every wave wait for all of its outstanding global
// loads (s_waitcnt vmcnt(0)) and so defeats loads prefetched stages ahead;
// here only the LDS writes must be complete before the barrier.
__device__ __forceinline__ void lds_sync() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Jet carries through tanh of one (point, column); index k runs over the
// streams: value, d/dx_1..d/dx_ND1, d^2/dx_1^2..d^2/dx_ND2^2.
// Forward: pre-activations in, activations out.
template <int ND1, int ND2, bool X64 = false>
__device__ __forceinline__ void jet_fwd(float* v) {
  float tt, s;
  tanh_pair<X64>(v[0], tt, s);
  const float sp = -2.0f * tt * s;
#pragma unroll
  for (int i = 0; i < ND2; ++i) v[1 + ND1 + i] = s * v[1 + ND1 + i] + sp * v[1 + i] * v[1 + i];
#pragma unroll
  for (int i = 0; i < ND1; ++i) v[1 + i] *= s;
  v[0] = tt;
}

// Reverse: activation cotangents in, pre-activation cotangents out, given the
// saved pre-activations ap.
template <int ND1, int ND2, bool X64 = false>
__device__ __forceinline__ void jet_bwd(float* g, const float* ap) {
  float tt, s;
  tanh_pair<X64>(ap[0], tt, s);
  const float sp = -2.0f * tt * s;
  const float spp = 2.0f * s * (3.0f * tt * tt - 1.0f);
  float ga = s * g[0];
#pragma unroll
  for (int i = 0; i < ND1; ++i) ga += sp * ap[1 + i] * g[1 + i];
#pragma unroll
  for (int i = 0; i < ND2; ++i) ga += (sp * ap[1 + ND1 + i] + spp * ap[1 + i] * ap[1 + i]) * g[1 + ND1 + i];
#pragma unroll
  for (int i = 0; i < ND1; ++i) {
    float v = s * g[1 + i];
    if (i < ND2) v += 2.0f * sp * ap[1 + i] * g[1 + ND1 + i];
    g[1 + i] = v;
  }
#pragma unroll
  for (int i = 0; i < ND2; ++i) g[1 + ND1 + i] *= s;
  g[0] = ga;
}

// Wait until at most N vector-memory operations of this wave are outstanding
// (N is an immediate).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// NS > 0 (16-bit types): the operand stages move from global memory straight
// into an NS-deep LDS ring (global_load_lds_dwordx4, no register staging),
// issued NS - 1 stages ahead of the multiply, so that the load latency is
// covered by several stages of matrix-core work.
// PM (fp32 storage only): products from bf16 pieces of the fp32 operands
// (ProdMode); PM_SPLIT3 folds the accumulators into fp64 after every stage.
// p.kx > 0 (two-term weights): operand X is kx wide and is read twice, the
// weight rows are 2 kx wide.
template <class T, int ND1, int ND2, int WM, int WN, int MT, int NT, int EPI, int OCC, bool DB = (OCC >= 2),
          int NS = 0, int PM = PM_NATIVE, int NB = 2>
__global__ void __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu(OCC)))
k_gemm_nt(const NtArgs<T> p) {
  constexpr int C = 1 + ND1 + ND2;
  constexpr int BM = 32 * MT * WM;
  constexpr int BN = 32 * NT * WN;
  constexpr int NTH = 64 * WM * WN;
  constexpr int ES = (int)sizeof(T);
  constexpr int KS = 64 / ES;                      // k values per stage
  constexpr int NCH = 64 / (16 * ES);              // 16-wide chunks per stage
  constexpr int ROWS = C * BM + BN;
  constexpr int STAGE = ROWS * LDS_PITCH;          // bytes of one operand stage
  constexpr int PIECES = ROWS * 4;
  constexpr int PPT = (PIECES + NTH - 1) / NTH;
  constexpr int OPITCH = BN * ES + 16;             // epilogue staging pitch (bytes)
  constexpr int OUTB = BM * OPITCH;
  constexpr int RING = (NS > 0 ? NS : 2) * STAGE;
  constexpr int LDSB = RING > OUTB ? RING : OUTB;
  static_assert(NS == 0 || (ES == 2 && NS >= 2 && ROWS % 16 == 0), "direct-to-LDS stages: 16-bit types");
  static_assert(PM == PM_NATIVE || ES == 4, "split products: fp32 storage");
  // fp32 mode (fp32 storage, products not split into bf16): tanh in fp64
  constexpr bool X64 = ES == 4 && PM != PM_SPLIT2 && PM != PM_SPLIT3;
  typedef typename Elem<T>::frag frag;
  __shared__ __attribute__((aligned(16))) char lds[LDSB];

  const int g = blockIdx.z;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % WM;
  const int wn = wave / WM;
  // logical tile: column tiles fastest, so the blocks reading one tile of
  // activations run together on one XCD and share it through its L2
  const int ntn = (p.N + BN - 1) / BN;
  const int64_t lt = xcd_remap(blockIdx.x, gridDim.x);
  const int64_t m0 = (lt / ntn) * BM;
  const int n0 = (int)(lt % ntn) * BN;
  const int64_t npts = p.seg.n_points;

  const char* Xb = (const char*)(p.X + g * p.x_g);
  const char* Wb = (const char*)(p.Wm + g * p.w_g);

  // each thread moves PPT 16-byte pieces of every stage: operand row piece>>2,
  // 16-byte segment piece&3 of its 64-byte k-slice.  The register ring
  // (NB > 2) loads unconditionally, so that the compiler can count the loads
  // in flight and wait only for the stage it stores (a load under a condition
  // makes it wait for all of them): points past the segment end and columns
  // past N read a clamped (valid) row, whose products are never stored, and
  // threads without a piece re-read the operand's first segment and drop it.
  // (Elsewhere the loads stay conditional: unconditional ones there moved the
  // staging registers of many kernels to scratch memory.)
  constexpr bool UNCOND = DB && NB > 2;
  const char* src[PPT];
  bool valid[PPT], isx[PPT];
#pragma unroll
  for (int i = 0; i < (NS > 0 ? 0 : PPT); ++i) {
    const int piece = tid + i * NTH;
    const int row = piece >> 2, sg = piece & 3;
    valid[i] = UNCOND;
    isx[i] = row < C * BM || piece >= PIECES;   // a dropped re-read stays inside X's first row
    src[i] = Xb;
    if (piece < PIECES) {
      if (row < C * BM) {
        const int k = row / BM, pp = row % BM;
        int64_t pt = m0 + pp;
        valid[i] = UNCOND || pt < npts;
        if (UNCOND && pt > npts - 1) pt = npts - 1;
        src[i] = Xb + (p.seg.row0 + k * p.seg.plane + pt) * p.ldx * (int64_t)ES + sg * 16;
      } else {
        int n = n0 + row - C * BM;
        valid[i] = UNCOND || n < p.N;
        if (UNCOND && n > p.N - 1) n = p.N - 1;
        src[i] = Wb + (int64_t)n * p.ldw * (int64_t)ES + sg * 16;
      }
    }
  }

  f32x16 acc[MT][C][NT];
#pragma unroll
  for (int u = 0; u < MT; ++u)
#pragma unroll
    for (int k = 0; k < C; ++k)
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[u][k][t][r] = 0.0f;

  // stage kt of the weights is stage kxs(kt) of operand X (two-term weights
  // read X twice)
  const int nk = p.K / KS;
  const int nkx = p.kx > 0 ? p.kx / KS : nk;
  auto kxs = [&](int kt) { return kt >= nkx ? kt - nkx : kt; };
  auto gload = [&](uint4* buf, int kt) {
    const int ktx = kxs(kt);
#pragma unroll
    for (int i = 0; i < PPT; ++i)
      buf[i] = (UNCOND || valid[i]) ? *(const uint4*)(src[i] + (int64_t)(isx[i] ? ktx : kt) * 64)
                                    : make_uint4(0u, 0u, 0u, 0u);
  };
  // PM_SPLIT2: each fp32 value of operand X is cut into its two bf16 pieces
  // once, as the stage is stored: a 64-byte stage row (16 k) then holds the
  // high pieces in segments 0-1 and the low pieces in segments 2-3, i.e. the
  // layout of a 16-bit stage whose first 16-wide chunk is the high part and
  // second the low part.  The weight rows arrive in that layout already (the
  // weight copies are split once per step), and are stored as loaded.
  auto lstore = [&](const uint4* buf, int stage) {
    char* base = lds + stage * STAGE;
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int piece = tid + i * NTH;
      if (piece >= PIECES) continue;
      const int row = piece >> 2, sg = piece & 3;
      if (PM == PM_SPLIT2 && row < C * BM) {
        const float* v = (const float*)&buf[i];
        bf16 hi[4], lo[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          hi[e] = (bf16)v[e];
          lo[e] = (bf16)(v[e] - (float)hi[e]);
        }
        *(uint2*)(base + lds_seg(row, sg >> 1) + (sg & 1) * 8) = __builtin_bit_cast(uint2, hi);
        *(uint2*)(base + lds_seg(row, 2 + (sg >> 1)) + (sg & 1) * 8) = __builtin_bit_cast(uint2, lo);
      } else {
        *(uint4*)(base + lds_seg(row, sg)) = buf[i];
      }
    }
  };
  // a fragment: 8 consecutive k of one row (16 bytes in 16-bit types, two
  // segments in fp32); every fragment row base is a multiple of 32, so the
  // segment swizzle of the lane's row is (lane >> 2) & 3
  const int gsw = (lane >> 2) & 3;
  bool odd = false;   // PM_SPLIT3: operand X negated in this stage
  auto frag_at = [&](const char* base, int row, int c) {
    if constexpr (ES == 2) {
      const int seg = 2 * c + (lane >> 5);
      return *(const frag*)(base + row * LDS_PITCH + ((seg ^ gsw) << 4));
    } else {
      const int seg = 2 * (lane >> 5);
      const u32x4 lo = *(const u32x4*)(base + row * LDS_PITCH + ((seg ^ gsw) << 4));
      const u32x4 hi = *(const u32x4*)(base + row * LDS_PITCH + (((seg + 1) ^ gsw) << 4));
      const u32x8 w = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      return __builtin_bit_cast(frag, w);
    }
  };
  // the high (c = 0) or low (c = 1) bf16 pieces of a PM_SPLIT2 fragment
  auto piece_at = [&](const char* base, int row, int c) {
    return *(const bf16x8*)(base + row * LDS_PITCH + (((2 * c + (lane >> 5)) ^ gsw) << 4));
  };
  auto compute = [&](int stage) {
    const char* base = lds + stage * STAGE;
    if constexpr (PM == PM_SPLIT2) {
      bf16x8 bp[NT][2];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int c = 0; c < 2; ++c) bp[t][c] = piece_at(base, C * BM + 32 * (wn * NT + t) + (lane & 31), c);
#pragma unroll
      for (int u = 0; u < MT; ++u)
#pragma unroll
        for (int k = 0; k < C; ++k) {
          bf16x8 ap[2];
#pragma unroll
          for (int c = 0; c < 2; ++c) ap[c] = piece_at(base, k * BM + 32 * (MT * wm + u) + (lane & 31), c);
#pragma unroll
          for (int t = 0; t < NT; ++t) mma_split<2>(acc[u][k][t], bp[t], ap);
        }
      return;
    }
    if constexpr (PM != PM_NATIVE) {
      // PM_SPLIT3: fp32 fragments (one chunk per stage), each cut into bf16
      // pieces as it is read.  PM_SPLIT3 negates operand X on every other stage (the fold subtracts
      // those stages): the matrix core's sums carry a small bias of one sign
      // whatever the sign of the result, which then cancels in the fp64 sum
      // instead of adding up over the stages.
      constexpr int NP = PM == PM_SPLIT3 ? 3 : 2;
      bf16x8 bp[NT][NP];
#pragma unroll
      for (int t = 0; t < NT; ++t) split_frag<NP>(frag_at(base, C * BM + 32 * (wn * NT + t) + (lane & 31), 0), bp[t]);
#pragma unroll
      for (int u = 0; u < MT; ++u)
#pragma unroll
        for (int k = 0; k < C; ++k) {
          bf16x8 ap[NP];
          f32x8 xf = frag_at(base, k * BM + 32 * (MT * wm + u) + (lane & 31), 0);
          if (PM == PM_SPLIT3 && odd) xf = -xf;
          split_frag<NP>(xf, ap);
#pragma unroll
          for (int t = 0; t < NT; ++t) mma_split<NP>(acc[u][k][t], bp[t], ap);
        }
      return;
    }
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      frag bfr[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) bfr[t] = frag_at(base, C * BM + 32 * (wn * NT + t) + (lane & 31), c);
#pragma unroll
      for (int u = 0; u < MT; ++u)
#pragma unroll
        for (int k = 0; k < C; ++k) {
          const frag afr = frag_at(base, k * BM + 32 * (MT * wm + u) + (lane & 31), c);
#pragma unroll
          for (int t = 0; t < NT; ++t) Elem<T>::mma(acc[u][k][t], bfr[t], afr);   // rows: columns n; cols: points
        }
    }
  };
  // PM_F64 (one fragment per wave and stream: 32 points x 32 columns, 2 x 2
  // blocks of the 16 x 16 fp64 product, whose lane l holds rows
  // (l >> 4) + 4 r and column l & 15 of a block)
  static_assert(PM != PM_F64 || (MT == 1 && NT == 1 && C <= 2), "fp64 products: one fragment per wave");
  f64x4 accd[PM == PM_F64 ? C : 1][2][2];
  if constexpr (PM == PM_F64) {
#pragma unroll
    for (int k = 0; k < C; ++k)
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) accd[k][a][b] = f64x4{0.0, 0.0, 0.0, 0.0};
  }
  // fp32 element kx (0..15) of LDS stage row r
  auto lds_f = [&](const char* base, int r, int kx) {
    return (double)*(const float*)(base + lds_seg(r, kx >> 2) + (kx & 3) * 4);
  };
  auto compute64 = [&](int stage) {
    const char* base = lds + stage * STAGE;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int kx = 4 * kk + (lane >> 4);
      double wv[2];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) wv[nb] = lds_f(base, C * BM + 32 * wn + 16 * nb + (lane & 15), kx);
#pragma unroll
      for (int k = 0; k < C; ++k)
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) {
          const double xv = lds_f(base, k * BM + 32 * wm + 16 * pb + (lane & 15), kx);
#pragma unroll
          for (int nb = 0; nb < 2; ++nb)
            accd[k][nb][pb] = __builtin_amdgcn_mfma_f64_16x16x4f64(wv[nb], xv, accd[k][nb][pb], 0, 0, 0);
        }
    }
  };
  // PM_SPLIT3: the stage's fp32 sums are added into (odd stages: subtracted
  // from) fp64 accumulators
  constexpr int A64 = PM == PM_SPLIT3 ? 1 : 0;
  double acc64[A64 ? MT : 1][A64 ? C : 1][A64 ? NT : 1][A64 ? 16 : 1];
  if constexpr (A64) {
#pragma unroll
    for (int u = 0; u < MT; ++u)
#pragma unroll
      for (int k = 0; k < C; ++k)
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc64[u][k][t][r] = 0.0;
  }
  auto fold = [&]() {
    if constexpr (A64) {
#pragma unroll
      for (int u = 0; u < MT; ++u)
#pragma unroll
        for (int k = 0; k < C; ++k)
#pragma unroll
          for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              acc64[u][k][t][r] += odd ? -(double)acc[u][k][t][r] : (double)acc[u][k][t][r];
              acc[u][k][t][r] = 0.0f;
            }
      odd = !odd;
    }
  };

  if constexpr (NS > 0) {
    // One DMA instruction of a wave fills 1 KB of LDS, lane l at byte 16 l:
    // 16 stage rows (row 16 g + l / 4, physical segment l % 4, holding the
    // logical segment (l % 4) ^ ((row >> 2) & 3) of the swizzled layout).
    // The NG row groups of a stage are dealt to the waves round-robin; a wave
    // with fewer groups repeats its last one (identical data to identical
    // bytes), so that every wave issues GPW loads per stage and one
    // immediate vmcnt fits all.  Points past the segment end and columns past
    // N read a clamped (valid) row: their products are never stored.
    constexpr int NG = ROWS / 16;
    constexpr int GPW = (NG + NTH / 64 - 1) / (NTH / 64);
    static_assert((NS - 2) * GPW <= 63, "outstanding loads exceed the vmcnt range");
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const char* dsrc[GPW];
    int dlds[GPW];
    bool dx[GPW];
#pragma unroll
    for (int i = 0; i < GPW; ++i) {
      int grp = wv + i * (NTH / 64);
      if (grp > NG - 1) grp = NG - 1;
      dlds[i] = grp * 1024;
      const int row = grp * 16 + (lane >> 2);
      const int ls = (lane & 3) ^ ((row >> 2) & 3);
      dx[i] = grp * 16 < C * BM;   // a 16-row group is all X rows or all weight rows (C * BM % 16 == 0)
      if (row < C * BM) {
        const int k = row / BM, pp = row % BM;
        int64_t pt = m0 + pp;
        if (pt > npts - 1) pt = npts - 1;
        dsrc[i] = Xb + (p.seg.row0 + k * p.seg.plane + pt) * p.ldx * (int64_t)ES + ls * 16;
      } else {
        int n = n0 + row - C * BM;
        if (n > p.N - 1) n = p.N - 1;
        dsrc[i] = Wb + (int64_t)n * p.ldw * (int64_t)ES + ls * 16;
      }
    }
    auto issue = [&](int kt, int stage) {
      const int ktx = kxs(kt);
#pragma unroll
      for (int i = 0; i < GPW; ++i)
        __builtin_amdgcn_global_load_lds((const void*)(dsrc[i] + (int64_t)(dx[i] ? ktx : kt) * 64),
                                         (lds_ptr_t)(lds + stage * STAGE + dlds[i]), 16, 0, 0);
    };
#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
      if (s < nk) issue(s, s);
    int st = 0;
    for (int kt = 0; kt < nk; ++kt) {
      // own loads of stage kt complete: the later stages issued so far may
      // still be in flight
      const int later = nk - 1 - kt;
      if constexpr (NS >= 4) {
        if (later >= 2) wait_vmcnt<2 * GPW>();
        else if (later == 1) wait_vmcnt<GPW>();
        else wait_vmcnt<0>();
      } else if constexpr (NS == 3) {
        if (later >= 1) wait_vmcnt<GPW>();
        else wait_vmcnt<0>();
      } else {
        wait_vmcnt<0>();
      }
      // every wave's loads of stage kt have landed, and every wave is done
      // with stage kt - 1, whose buffer the next issue refills
      lds_sync();
      if (kt + NS - 1 < nk) issue(kt + NS - 1, st == 0 ? NS - 1 : st - 1);
      if constexpr (PM == PM_F64) compute64(st); else compute(st);
      fold();
      st = st + 1 == NS ? 0 : st + 1;
    }
    lds_sync();
  } else if constexpr (DB && NB > 2) {
    // two LDS stages and a ring of NB register buffers: buffer b holds the
    // stages kt = b (mod NB), so the global loads of stage kt + NB are issued
    // while stage kt is multiplied.  Loads are unconditional (stage index
    // clamped), so the compiler's waits are static counts.
    uint4 bufs[NB][PPT];
    const int last = nk - 1;
#pragma unroll
    for (int b = 0; b < NB; ++b) gload(bufs[b], b < last ? b : last);
    lstore(bufs[0], 0);
    gload(bufs[0], NB < last ? NB : last);
    lds_sync();
    // UR rounds of the ring per loop pass: the compiler drains every load in
    // flight once per pass (its wait analysis does not carry the ring across
    // the back edge), so longer passes drain less often
    constexpr int UR = 4;
    for (int k0 = 0; k0 < nk; k0 += NB * UR) {
#pragma unroll
      for (int u = 0; u < NB * UR; ++u) {
        const int kt = k0 + u;
        if (kt >= nk) break;
        if constexpr (PM == PM_F64) compute64(kt & 1); else compute(kt & 1);
        fold();
        __builtin_amdgcn_sched_barrier(0);
        if (kt + 1 < nk) lstore(bufs[(u + 1) % NB], (kt + 1) & 1);
        gload(bufs[(u + 1) % NB], kt + 1 + NB < last ? kt + 1 + NB : last);
        lds_sync();
      }
    }
  } else if constexpr (DB) {
    // two LDS stages, two register buffers: the global loads of stage kt+2
    // are issued before stage kt is multiplied; one barrier per stage
    // prefetches are unconditional (the stage index is clamped; loads past
    // the last stage are never stored): conditional loads would force
    // register copies that wait for the data
    uint4 b0[PPT], b1[PPT];
    gload(b0, 0);
    lstore(b0, 0);
    gload(b1, nk > 1 ? 1 : 0);
    lds_sync();
    for (int kt = 0; kt < nk; kt += 2) {
      gload(b0, kt + 2 < nk ? kt + 2 : nk - 1);
      if constexpr (PM == PM_F64) compute64(0); else compute(0);
      fold();
      __builtin_amdgcn_sched_barrier(0);
      if (kt + 1 < nk) lstore(b1, 1);
      lds_sync();
      if (kt + 1 >= nk) break;
      gload(b1, kt + 3 < nk ? kt + 3 : nk - 1);
      if constexpr (PM == PM_F64) compute64(1); else compute(1);
      fold();
      __builtin_amdgcn_sched_barrier(0);
      if (kt + 2 < nk) lstore(b0, 0);
      lds_sync();
    }
  } else {
    // large tiles (one wave per SIMD): two LDS stages, one register buffer
    // loaded one stage ahead
    uint4 b0[PPT];
    gload(b0, 0);
    lstore(b0, 0);
    lds_sync();
    for (int kt = 0; kt < nk; ++kt) {
      gload(b0, kt + 1 < nk ? kt + 1 : nk - 1);
      if constexpr (PM == PM_F64) compute64(kt & 1); else compute(kt & 1);
      fold();
      __builtin_amdgcn_sched_barrier(0);
      if (kt + 1 < nk) lstore(b0, (kt + 1) & 1);
      lds_sync();
    }
  }
  if constexpr (A64) {
#pragma unroll
    for (int u = 0; u < MT; ++u)
#pragma unroll
      for (int k = 0; k < C; ++k)
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[u][k][t][r] = (float)acc64[u][k][t][r];
  }
  if constexpr (PM == PM_F64) {
    // each stream through LDS, [point][column] floats (pitch 65), into the
    // lane layout of the fp32 fragments the epilogue reads
    float* tl = (float*)lds;
    lds_sync();
#pragma unroll
    for (int k = 0; k < C; ++k) {
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            tl[(32 * wm + 16 * pb + (lane & 15)) * 65 + 32 * wn + 16 * nb + (lane >> 4) + 4 * r] =
                (float)accd[k][nb][pb][r];
      lds_sync();
#pragma unroll
      for (int r = 0; r < 16; ++r)
        acc[0][k][0][r] = tl[(32 * wm + (lane & 31)) * 65 + 32 * wn + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)];
      lds_sync();
    }
  }

  // ---- epilogue.  The products were formed as W . X^T, so lane (lane & 31)
  // owns one point of each of its MT point sub-tiles and, in register group q
  // (regs 4q..4q+3), four consecutive columns 8q + 4*(lane >> 5) + 0..3 of
  // every 32x32 tile: all jet streams of a (point, column) sit in the same
  // lane.  Results are staged through LDS one stream at a time and leave in
  // full 16-byte row segments.
  const int hh = lane >> 5;
  auto mloc = [&](int u) { return 32 * (MT * wm + u) + (lane & 31); };            // point within the block
  auto ncol = [&](int t, int q) { return 32 * (wn * NT + t) + 8 * q + 4 * hh; };   // column within the block

  if (EPI == EPI_DF) {
    const int64_t ldY = p.sY_ld > 0 ? p.sY_ld : p.nY, ldU = p.sU_ld > 0 ? p.sU_ld : p.nU;
#pragma unroll
    for (int u = 0; u < MT; ++u) {
      const int64_t pt = m0 + mloc(u);
      if (pt >= npts) continue;
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int n = n0 + ncol(t, q) + e;
            const float v = p.df_sign * acc[u][0][t][4 * q + e];
            if (n < p.nY) p.seedY[g * p.sY_g + pt * ldY + n] = v;
            else if (n < p.nY + p.nU) p.seedU[g * p.sU_g + pt * ldU + p.sU_off + (n - p.nY)] = v;
          }
    }
    return;
  }

  // adds a [points x columns] array of every stream (rows laid out as the
  // outputs) to the accumulators: residual skips of a shared trunk
  auto add_rows = [&](const T* src) {
#pragma unroll
    for (int u = 0; u < MT; ++u) {
      const int64_t pt = m0 + mloc(u);
      const bool pvalid = pt < npts;
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int nb = n0 + ncol(t, q);
          if (!pvalid || nb >= p.N) continue;
#pragma unroll
          for (int k = 0; k < C; ++k) {
            float v[4];
            load4<T>(src + g * p.o_g + (p.seg.row0 + k * p.seg.plane + pt) * p.ldo + nb, v);
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[u][k][t][4 * q + e] += v[e];
          }
        }
    }
  };

  // staging: one [BM x BN] plane at a time through LDS, copied out in full
  // 16-byte row segments
  constexpr int CPR = BN * ES / 16;                // 16-byte chunks per staged row
  constexpr int CHUNKS = BM * CPR;
  auto stage_out = [&](int k, T* dst) {
#pragma unroll
    for (int u = 0; u < MT; ++u)
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[u][k][t][4 * q + e];
          store4<T>((T*)(lds + mloc(u) * OPITCH + ncol(t, q) * ES), v);
          __builtin_amdgcn_sched_barrier(0);
        }
    lds_sync();
#pragma unroll
    for (int it = 0; it < (CHUNKS + NTH - 1) / NTH; ++it) {
      const int i = tid + it * NTH;
      if (CHUNKS % NTH != 0 && i >= CHUNKS) break;
      const int row = i / CPR, ch = i % CPR;
      const int64_t ptr = m0 + row;
      const int n = n0 + ch * (16 / ES);
      if (ptr < npts && n < p.N)
        *(uint4*)(dst + g * p.o_g + (p.seg.row0 + k * p.seg.plane + ptr) * p.ldo + n) =
            *(const uint4*)(lds + row * OPITCH + ch * 16);
    }
    lds_sync();
  };

  if (EPI == EPI_FWD) {
    // pre-activations (bias on the value stream), then activations in place:
    //   h = t, h'_i = s a'_i, h''_i = s a''_i + s' (a'_i)^2
#pragma unroll
    for (int u = 0; u < MT; ++u)
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          // columns past N take the last bias (their results are never stored)
          const int n = n0 + ncol(t, r >> 2) + (r & 3);
          if (p.bias) acc[u][0][t][r] += p.bias[g * p.b_g + (n < p.N ? n : p.N - 1)];
        }
    if (p.out_a) {
#pragma unroll
      for (int k = 0; k < C; ++k) stage_out(k, p.out_a);
    }
#pragma unroll
    for (int u = 0; u < MT; ++u)
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float v[C];
#pragma unroll
          for (int k = 0; k < C; ++k) v[k] = acc[u][k][t][r];
          jet_fwd<ND1, ND2, X64>(v);
#pragma unroll
          for (int k = 0; k < C; ++k) acc[u][k][t][r] = v[k];
        }
    // residual block output: h_l = tanh carry + h_{l-2}, stream by stream
    if (p.skip) add_rows(p.skip);
#pragma unroll
    for (int k = 0; k < C; ++k) stage_out(k, p.out_h);
    return;
  }

  // skip cotangent of a residual block's input, and the total kept for the
  // skip below it
  if (p.skip_g) add_rows(p.skip_g);
  if (p.out_gh) {
#pragma unroll
    for (int k = 0; k < C; ++k) stage_out(k, p.out_gh);
  }

  // reverse carry, in place: acc[k] becomes the cotangent of the saved
  // pre-activation a_k of the layer below
#pragma unroll
  for (int u = 0; u < MT; ++u) {
    // points past the segment end and columns past N read a clamped (valid)
    // element: their results are never stored, and unconditional loads keep
    // the loads of a fragment together, without a branch around each
    int64_t pt = m0 + mloc(u);
    if (pt > npts - 1) pt = npts - 1;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      // the saved pre-activations of all four column groups of this fragment,
      // issued together (one memory latency per fragment, not per group)
      typedef typename std::conditional<ES == 2, uint2, float4>::type raw_t;
      raw_t raw[4][C];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        int nb = n0 + ncol(t, q);
        if (nb >= p.N) nb = 0;
#pragma unroll
        for (int k = 0; k < C; ++k)
          raw[q][k] = *(const raw_t*)(p.aprev + g * p.o_g + (p.seg.row0 + k * p.seg.plane + pt) * p.ldo + nb);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float ap[C][4];
#pragma unroll
        for (int k = 0; k < C; ++k) {
          if constexpr (ES == 2) {
            const T* ev = (const T*)&raw[q][k];
#pragma unroll
            for (int e = 0; e < 4; ++e) ap[k][e] = Elem<T>::to_f(ev[e]);
          } else {
            ap[k][0] = raw[q][k].x; ap[k][1] = raw[q][k].y; ap[k][2] = raw[q][k].z; ap[k][3] = raw[q][k].w;
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * q + e;
          float gv[C], av[C];
#pragma unroll
          for (int k = 0; k < C; ++k) {
            gv[k] = acc[u][k][t][r];
            av[k] = ap[k][e];
          }
          jet_bwd<ND1, ND2, X64>(gv, av);
#pragma unroll
          for (int k = 0; k < C; ++k) acc[u][k][t][r] = gv[k];
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#pragma unroll
  for (int k = 0; k < C; ++k) stage_out(k, p.out_da);
}

// ---------------------------------------------------------------------------
// k_gemm_nt_wr: the products and epilogues of k_gemm_nt for 16-bit storage
// and K = N = 128 (hidden layers of width 128), as a persistent kernel
// built to keep HBM busy.  Each block copies the weight matrix into LDS once
// and then walks tiles of 32 points (all jet streams, the whole K extent at
// once).  While one tile is multiplied and written out, the activations of
// its successor (and, in the reverse pass, the saved pre-activations of the
// tile itself) are already on their way into registers, so every block keeps
// a whole tile of loads in flight.  Four waves; wave w owns columns
// 32w..32w+31 of every stream.  SKIP: the residual blocks of a shared trunk
// (forward: h_l += h_{l-2}; reverse: the block's skip cotangent added, the
// total kept), read like the saved pre-activations, ahead of the prefetch.
// ---------------------------------------------------------------------------
// one block per CU (and the whole register file) for the skip variant of
// five streams, whose skip rows do not fit beside the prefetch otherwise
template <int C, bool SKIP, bool TWO = false>
constexpr int wr_blocks_per_cu() { return (SKIP || TWO) && C >= 5 ? 1 : 2; }

// TWO: two-term weight rows [W_hi | W_lo] (forward, K = 2 x 128): W_hi is the
// LDS-resident tile, each wave keeps its columns' W_lo fragments in registers
// for the whole launch.
template <class T, int ND1, int ND2, int EPI, bool FIRST, bool SKIP = false, bool TWO = false>
__global__ void __launch_bounds__(256)
__attribute__((amdgpu_waves_per_eu(wr_blocks_per_cu<1 + ND1 + ND2, SKIP, TWO>())))
k_gemm_nt_wr(const NtArgs<T> p, int64_t ntiles) {
  static_assert(sizeof(T) == 2, "16-bit storage only");
  static_assert(!(SKIP && FIRST), "residual blocks never start at the first layer");
  static_assert(!TWO || EPI == EPI_FWD, "two-term weights: forward products only");
  constexpr int C = 1 + ND1 + ND2;
  constexpr int BM = 32, BN = 128, NTH = 256, ES = 2;
  constexpr int RB = 256;                          // bytes of one operand row (K = 128)
  constexpr int PITCH = RB + 16;                   // LDS row pitch: conflict-free 16-byte fragment reads
  constexpr int WREG = BN * PITCH;                 // weight tile
  constexpr int XREG = C * BM * PITCH;             // activation tile, reused to stage the outputs
  constexpr int OPITCH = BN * ES + 16;             // staging pitch of one output plane
  static_assert(C * BM * OPITCH <= XREG, "staging must fit in the activation region");
  constexpr int SEGS = RB / 16;                    // 16-byte pieces per row
  constexpr int XP = C * BM * SEGS / NTH;          // pieces per thread of an activation tile
  constexpr int WP = BN * SEGS / NTH;              // pieces per thread of the weights
  constexpr int RPP = NTH / SEGS;                  // rows covered by one piece index
  typedef typename Elem<T>::frag frag;
  constexpr int W1REG = FIRST ? BN * 4 * 4 : 0;   // W1 columns 0..2 of every unit (fp32, padded to 4)
  __shared__ __attribute__((aligned(16))) char lds[WREG + XREG + W1REG];
  char* const wl = lds;
  char* const xl = lds + WREG;
  float* const w1l = (float*)(lds + WREG + XREG);

  const int g = blockIdx.z;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int hh = lane >> 5;
  const int sg = tid % SEGS;
  const int64_t npts = p.seg.n_points;
  const char* Xb = (const char*)(p.X + g * p.x_g);
  const char* Wb = (const char*)(p.Wm + g * p.w_g);

  // weights (N = 128 rows)
  {
    u32x4 wb[WP];
#pragma unroll
    for (int i = 0; i < WP; ++i) wb[i] = *(const u32x4*)(Wb + (int64_t)(tid / SEGS + RPP * i) * p.ldw * ES + sg * 16);
#pragma unroll
    for (int i = 0; i < WP; ++i) *(u32x4*)(wl + (tid / SEGS + RPP * i) * PITCH + sg * 16) = wb[i];
  }
  // the low terms of the wave's 32 weight rows, one fragment per 16-wide k chunk
  frag wlo[TWO ? RB / 32 : 1];
  if constexpr (TWO) {
    const char* wrow = Wb + (int64_t)(32 * wave + (lane & 31)) * p.ldw * ES + RB;
#pragma unroll
    for (int c = 0; c < RB / 32; ++c) wlo[c] = *(const frag*)(wrow + c * 32 + hh * 16);
  }

  // first layer formed in the kernel: W1[n][0..d-1] for every unit n
  if constexpr (FIRST) {
    if (tid < BN) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        w1l[tid * 4 + i] = i < p.f_d ? p.fp1[g * p.fp_g + (int64_t)tid * p.f_in + i] : 0.0f;
    }
    lds_sync();
  }
  // sample and coordinate row of point pt of the segment
  auto f_sample = [&](int64_t pt) { return pt / p.fPn; };
  auto f_xrow = [&](int64_t pt) { return p.fx_shared ? pt % p.fPn : pt; };

  // activation rows of a tile; points past the end repeat the last point.
  // Stream bases are uniform (scalar); a thread's two point rows are 32-bit
  // byte offsets (the host checks that a stream plane spans < 2^31 bytes).
  static_assert(BM == 2 * RPP, "two point rows per thread");
  constexpr bool GENX = FIRST && EPI == EPI_FWD;   // forward: X is the first layer's activations
  constexpr int XPR = GENX ? 1 : XP;
  u32x4 xb[XPR];
  // first layer: the thread's two points (rows tid / SEGS + RPP j) and its 8
  // units 8 sg..8 sg+7: coordinates and z-projection of the next tile
  float fxv[2][3], fzv[2][8];
  auto xload = [&](int64_t tile) {
    int64_t p0 = tile * BM + tid / SEGS, p1 = p0 + RPP;
    if (p0 >= npts) p0 = npts - 1;
    if (p1 >= npts) p1 = npts - 1;
    if constexpr (GENX) {
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int64_t pt = jj ? p1 : p0;
        const float* xv = p.fx + g * p.fx_g + f_xrow(pt) * p.f_d;
#pragma unroll
        for (int i = 0; i < 3; ++i) fxv[jj][i] = i < p.f_d ? xv[i] : 0.0f;
        const float4* zv = (const float4*)(p.fzp + g * p.fzp_g + f_sample(pt) * BN + 8 * sg);
        const float4 z0 = zv[0], z1 = zv[1];
        fzv[jj][0] = z0.x; fzv[jj][1] = z0.y; fzv[jj][2] = z0.z; fzv[jj][3] = z0.w;
        fzv[jj][4] = z1.x; fzv[jj][5] = z1.y; fzv[jj][6] = z1.z; fzv[jj][7] = z1.w;
      }
    } else {
      const uint32_t o0 = (uint32_t)(p0 * p.ldx * ES) + sg * 16, o1 = (uint32_t)(p1 * p.ldx * ES) + sg * 16;
#pragma unroll
      for (int i = 0; i < XP; ++i) {
        const char* base = Xb + (p.seg.row0 + (i >> 1) * p.seg.plane) * p.ldx * ES;
        xb[i] = *(const u32x4*)(base + ((i & 1) ? o1 : o0));
      }
    }
  };
  auto ncol = [&](int q) { return 32 * wave + 8 * q + 4 * hh; };   // first of the lane's 4 columns in group q

  // bias and output weights of the lane's 16 columns (fixed for the launch)
  float bias[16], wo[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) bias[r] = wo[r] = 0.0f;
  float bout = 0.0f;
  if (EPI == EPI_FWD && p.bias) {
#pragma unroll
    for (int r = 0; r < 16; ++r) bias[r] = p.bias[g * p.b_g + ncol(r >> 2) + (r & 3)];
  }
  if (!SKIP && EPI == EPI_FWD && p.y) {           // (the output layer is never fused with a skip)
#pragma unroll
    for (int r = 0; r < 16; ++r) wo[r] = p.wout[g * p.wo_g + ncol(r >> 2) + (r & 3)];
    bout = p.wout[g * p.wo_g + BN];
  }

  auto pack8 = [&](const float* v) {
    u32x4 w;
#pragma unroll
    for (int h2 = 0; h2 < 4; ++h2) {
      const T lo = Elem<T>::from_f(v[2 * h2]), hi = Elem<T>::from_f(v[2 * h2 + 1]);
      w[h2] = (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
    }
    return w;
  };
  auto xstore = [&](int64_t tile) {
    if constexpr (GENX) {
      // first layer, as in the standalone kernel: a = zproj + sum_i W1[:, i] x_i,
      // h = t, h'_i = s W1[:, i], h''_i = s' W1[:, i]^2 (a' = W1[:, i], a'' = 0)
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        int64_t pt = tile * BM + tid / SEGS + RPP * jj;
        if (pt >= npts) pt = npts - 1;
        float a[8], hv[8], s8[8], sp8[8], fwc[3][8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float4 w4 = *(const float4*)(w1l + (8 * sg + e) * 4);
          fwc[0][e] = w4.x; fwc[1][e] = w4.y; fwc[2][e] = w4.z;
          a[e] = fzv[jj][e];
#pragma unroll
          for (int i = 0; i < 3; ++i) a[e] += fwc[i][e] * fxv[jj][i];
          float t, sd;
          tanh_ts(a[e], t, sd);
          hv[e] = t;
          s8[e] = sd;
          sp8[e] = -2.0f * t * sd;
        }
        const int row = tid / SEGS + RPP * jj;
#pragma unroll
        for (int k = 0; k < C; ++k) {
          float v[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            if (k == 0) v[e] = hv[e];
            else if (k <= ND1) v[e] = s8[e] * fwc[k - 1][e];
            else v[e] = sp8[e] * fwc[k - 1 - ND1][e] * fwc[k - 1 - ND1][e];
          }
          const u32x4 w = pack8(v);
          *(u32x4*)(xl + (k * BM + row) * PITCH + sg * 16) = w;
          if (p.f_out_h)                           // past the end: the last point's values again
            *(u32x4*)(p.f_out_h + g * p.o_g + (p.seg.row0 + k * p.seg.plane + pt) * p.ldo + 8 * sg) = w;
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < XP; ++i) *(u32x4*)(xl + (tid / SEGS + RPP * i) * PITCH + sg * 16) = xb[i];
    }
  };

  // The activations of a tile go from registers to LDS at the end of the
  // previous iteration, after its stores were issued: the wait for the
  // prefetch then leaves those stores in flight (the memory counter drains
  // in issue order, and the same operations are pending on every iteration).
  int64_t tile = blockIdx.x;
  xload(tile);
  xstore(tile);
  for (; tile < ntiles; tile += gridDim.x) {
    const int64_t m0 = tile * BM;
    lds_sync();

    // reverse pass: the saved pre-activations of this tile, in the lane
    // layout of the products (point lane & 31, four columns per group).
    // Issued before the prefetch so that waiting for them (the memory
    // counter drains in issue order) does not wait for the prefetch.
    u32x2 apr[FIRST ? 1 : C][4];
    float fzb[16], fxb[3];
    if (FIRST && EPI == EPI_BWD) {
      // first layer: z-projection of the lane's 16 units and its coordinates
      int64_t pt = m0 + (lane & 31);
      if (pt >= npts) pt = npts - 1;
      const float* zr = p.fzp + g * p.fzp_g + f_sample(pt) * BN;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 z4 = *(const float4*)(zr + ncol(q));
        fzb[4 * q] = z4.x; fzb[4 * q + 1] = z4.y; fzb[4 * q + 2] = z4.z; fzb[4 * q + 3] = z4.w;
      }
      const float* xv = p.fx + g * p.fx_g + f_xrow(pt) * p.f_d;
#pragma unroll
      for (int i = 0; i < 3; ++i) fxb[i] = i < p.f_d ? xv[i] : 0.0f;
    } else if (EPI == EPI_BWD) {
      int64_t pt = m0 + (lane & 31);
      if (pt >= npts) pt = npts - 1;
      const uint32_t po = (uint32_t)(pt * p.ldo * ES);
#pragma unroll
      for (int k = 0; k < C; ++k) {
        const char* base = (const char*)(p.aprev + g * p.o_g + (p.seg.row0 + k * p.seg.plane) * p.ldo);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          apr[k][q] = *(const u32x2*)(base + po + ncol(q) * ES);
        }
      }
    }
    // residual skip of the tile in the same lane layout: the block input
    // h_{l-2} (forward) or the skip cotangent of a block input (reverse)
    u32x2 skp[SKIP ? C : 1][4];
    const T* const skip_src = EPI == EPI_FWD ? p.skip : p.skip_g;
    if (SKIP && skip_src) {
      int64_t pt = m0 + (lane & 31);
      if (pt >= npts) pt = npts - 1;
      const uint32_t po = (uint32_t)(pt * p.ldo * ES);
#pragma unroll
      for (int k = 0; k < (SKIP ? C : 1); ++k) {
        const char* base = (const char*)(skip_src + g * p.o_g + (p.seg.row0 + k * p.seg.plane) * p.ldo);
#pragma unroll
        for (int q = 0; q < 4; ++q) skp[k][q] = *(const u32x2*)(base + po + ncol(q) * ES);
      }
    }

    {
      const int64_t nx = tile + gridDim.x;
      xload(nx < ntiles ? nx : tile);              // unconditional: the last prefetch is never used
    }
    __builtin_amdgcn_sched_barrier(0);             // keep the loads ahead of the products

    f32x16 acc[C];
#pragma unroll
    for (int k = 0; k < C; ++k)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[k][r] = 0.0f;
    // register r of a lane holds column ncol(r / 4) + r % 4 of its point,
    // which is element r % 4 of the lane's u32x2 pair (r / 4)
    auto add_skip = [&]() {
#pragma unroll
      for (int k = 0; k < (SKIP ? C : 1); ++k)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const uint32_t w = skp[k][r >> 2][(r & 3) >> 1];
          const uint16_t h = (r & 1) ? (uint16_t)(w >> 16) : (uint16_t)(w & 0xffffu);
          acc[k][r] += Elem<T>::to_f(__builtin_bit_cast(T, h));
        }
    };
#pragma unroll
    for (int c = 0; c < RB / 32; ++c) {
      const int koff = c * 32 + hh * 16;
      const frag bfr = *(const frag*)(wl + (32 * wave + (lane & 31)) * PITCH + koff);
#pragma unroll
      for (int k = 0; k < C; ++k) {
        const frag afr = *(const frag*)(xl + (k * BM + (lane & 31)) * PITCH + koff);
        if constexpr (TWO) Elem<T>::mma(acc[k], wlo[c], afr);
        Elem<T>::mma(acc[k], bfr, afr);            // rows: columns n; cols: points
      }
    }
    __builtin_amdgcn_sched_barrier(0);             // no epilogue work (waits on the loads) above here
    lds_sync();                                    // the activation region is free for staging

    // all C output planes of the tile at once: stream k is staged in rows
    // [32k, 32k+32) of the (free) activation region, then copied out in
    // full 16-byte row segments
    auto stage_out = [&](T* dst) {
#pragma unroll
      for (int k = 0; k < C; ++k)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[k][4 * q + e];
          store4<T>((T*)(xl + (k * BM + (lane & 31)) * OPITCH + ncol(q) * ES), v);
        }
      lds_sync();
      // rows of points past the end hold exactly the values of the last
      // point (same inputs, same arithmetic): they are written over it
      // unconditionally, which keeps the memory counter static for the
      // prefetch waits
      constexpr int CPR = BN * ES / 16;            // 16-byte chunks per row
#pragma unroll
      for (int j = 0; j < C * BM * CPR / NTH; ++j) {
        const int i = tid + j * NTH;
        const int row = i / CPR, ch = i % CPR;
        const int k = row / BM;
        int64_t pt = m0 + row % BM;
        if (pt >= npts) pt = npts - 1;
        *(u32x4*)(dst + g * p.o_g + (p.seg.row0 + k * p.seg.plane + pt) * p.ldo + ch * (16 / ES)) =
            *(const u32x4*)(xl + row * OPITCH + ch * 16);
      }
      lds_sync();
    };

    if (EPI == EPI_FWD) {
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[0][r] += bias[r];
      if (p.out_a) {
        stage_out(p.out_a);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float v[C];
#pragma unroll
        for (int k = 0; k < C; ++k) v[k] = acc[k][r];
        jet_fwd<ND1, ND2>(v);
#pragma unroll
        for (int k = 0; k < C; ++k) acc[k][r] = v[k];
      }
      if constexpr (SKIP) {
        if (p.skip) add_skip();                    // residual block output
      }
      if (!SKIP && p.y) {
        // output layer: y = w_out . h over the activations as stored, summed
        // over the lane's columns, the two lane halves, then the four waves
        // in wave order (through LDS)
        float* red = (float*)xl;
#pragma unroll
        for (int k = 0; k < C; ++k) {
          float part = 0.0f;
#pragma unroll
          for (int r = 0; r < 16; ++r) part += wo[r] * Elem<T>::to_f(Elem<T>::from_f(acc[k][r]));
          part += __shfl_xor(part, 32);
          if (lane < 32) red[(wave * C + k) * 32 + lane] = part;
        }
        lds_sync();
        if (tid < C * 32) {
          const int k = tid >> 5, pp = tid & 31;
          float v = red[k * 32 + pp];
#pragma unroll
          for (int w = 1; w < 4; ++w) v += red[(w * C + k) * 32 + pp];
          if (k == 0) v += bout;
          int64_t pt = m0 + pp;
          if (pt >= npts) pt = npts - 1;             // past the end: the last point's value again
          p.y[g * p.y_g + p.seg.row0 + k * p.seg.plane + pt] = v;
        }
        lds_sync();
      }
      if (p.out_h) stage_out(p.out_h);
    } else {
      if constexpr (SKIP) {
        // skip cotangent of a residual block's input, and the total kept for
        // the skip below it (all loads of the tile were consumed before the
        // staging barrier, so an in-place total is safe)
        if (p.skip_g) add_skip();
        if (p.out_gh) stage_out(p.out_gh);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * q + e;
          float gv[C], av[C];
#pragma unroll
          for (int k = 0; k < C; ++k) gv[k] = acc[k][r];
          if constexpr (FIRST) {
            // the first layer's pre-activations as the standalone pass stores
            // them: a (rounded), a'_i = W1[n][i] (rounded), a''_i = 0
            const float* w1 = w1l + (ncol(q) + e) * 4;
            float a = fzb[r];
#pragma unroll
            for (int i = 0; i < 3; ++i) a += w1[i] * fxb[i];
            av[0] = Elem<T>::to_f(Elem<T>::from_f(a));
#pragma unroll
            for (int i = 0; i < ND1; ++i) av[1 + i] = Elem<T>::to_f(Elem<T>::from_f(w1[i]));
#pragma unroll
            for (int i = 0; i < ND2; ++i) av[1 + ND1 + i] = 0.0f;
          } else {
#pragma unroll
            for (int k = 0; k < C; ++k) {
              const uint32_t w = apr[k][q][e >> 1];
              const uint16_t h = (e & 1) ? (uint16_t)(w >> 16) : (uint16_t)(w & 0xffffu);
              av[k] = Elem<T>::to_f(__builtin_bit_cast(T, h));
            }
          }
          jet_bwd<ND1, ND2>(gv, av);
#pragma unroll
          for (int k = 0; k < C; ++k) acc[k][r] = gv[k];
        }
      }
      stage_out(p.out_da);
    }
    {
      const int64_t nx = tile + gridDim.x;
      xstore(nx < ntiles ? nx : tile);             // the next tile (the region is free again)
    }
  }
}

// ---------------------------------------------------------------------------
// dW[n][j] = sum_{rows m} dA[m][n] H[m][j]   (contraction over rows)
// Each block owns a (BNn x BJ) output tile and one contiguous range of rows.
// Row slices are transposed into LDS: every operand column is one 64-byte
// line of SR rows (8 rows per 16-byte fragment), so the fragments are single
// 16-byte reads.  Line base of column c (bytes): 80 c, plus 64 for columns
// 16..31 of every 32 (period 2624 bytes).  With lanes running over 16 row
// pairs x 4 column groups, each transposing write instruction then hits 64
// distinct banks, and the fragment reads stay conflict-free.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int dw_col(int c) {
  return (c >> 5) * 2624 + (c & 31) * 80 + ((c & 16) ? 64 : 0);
}

// PM (fp32 storage): products from bf16 pieces (ProdMode); with PM_SPLIT3
// the stage sums are folded into fp64 and the split partials are written in
// fp64 to partial64 (partial is unused).
template <class T, int WM, int WN, int NT, int OCC, int NB, int PM = PM_NATIVE>
__global__ void __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu(OCC)))
k_gemm_dw(const T* __restrict__ dA, int64_t a_g, int64_t lda, const T* __restrict__ H, int64_t h_g,
          int64_t ldh, int64_t R, int64_t n_value, int N, int J, float* __restrict__ partial,
          double* __restrict__ pdb, int n_split, int64_t rows_per_split, double* __restrict__ partial64) {
  static_assert(PM == PM_NATIVE || sizeof(T) == 4, "split products: fp32 storage");
  constexpr int BNn = 32 * NT * WM;
  constexpr int BJ = 32 * NT * WN;
  constexpr int NTH = 64 * WM * WN;
  constexpr int ES = (int)sizeof(T);
  constexpr int SR = 64 / ES;               // rows per stage
  constexpr int EPP = 16 / ES;              // elements per 16-byte load
  // PM_SPLIT2: every fp32 value is cut into its two bf16 pieces once, as the
  // stage is stored; a 64-byte column line (16 rows) then holds the 16 high
  // pieces followed by the 16 low pieces
  constexpr bool SPL = PM == PM_SPLIT2;
  constexpr int RPP = (ES == 2 || SPL) ? 2 : 1;   // rows per piece (packed 4-byte LDS writes)
  constexpr int NRP = SR / RPP;             // row pieces per stage (16)
  constexpr int NCH = 64 / (16 * ES);
  constexpr int PA = NRP * (BNn / EPP);
  constexpr int PB = NRP * (BJ / EPP);
  constexpr int PIECES = PA + PB;
  constexpr int PPT = (PIECES + NTH - 1) / NTH;
  constexpr int REGA = (BNn / 32) * 2624;   // bytes of the dA part of a stage
  constexpr int STAGE = REGA + (BJ / 32) * 2624;
  typedef typename Elem<T>::frag frag;
  __shared__ __attribute__((aligned(16))) char lds[2 * STAGE];

  // logical block: output tiles fastest, so the blocks reading one row range
  // run together on one XCD
  const int tiles_n = (N + BNn - 1) / BNn;
  const int tiles = tiles_n * ((J + BJ - 1) / BJ);
  const int64_t lb = xcd_remap(blockIdx.x, gridDim.x);
  const int tile = (int)(lb % tiles);
  const int tn = tile % tiles_n;
  const int tj = tile / tiles_n;
  const int split = (int)(lb / tiles);
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
  const int nst = (int)((r1 - r0 + SR - 1) / SR);

  const T* A = dA + g * a_g;
  const T* B = H + g * h_g;

  f32x16 acc[NT][NT];
#pragma unroll
  for (int a = 0; a < NT; ++a)
#pragma unroll
    for (int b = 0; b < NT; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;
  constexpr int A64 = PM == PM_SPLIT3 ? 1 : 0;
  double acc64[A64 ? NT : 1][A64 ? NT : 1][A64 ? 16 : 1];
  if constexpr (A64) {
#pragma unroll
    for (int a = 0; a < NT; ++a)
#pragma unroll
      for (int b = 0; b < NT; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc64[a][b][r] = 0.0;
  }
  // PM_F64: a wave's 32 x 32 outputs as 2 x 2 blocks of the 16 x 16 fp64
  // product (lane l: rows (l >> 4) + 4 r, column l & 15 of a block)
  static_assert(PM != PM_F64 || NT == 1, "fp64 products: one fragment per wave");
  f64x4 accd[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) accd[a][b] = f64x4{0.0, 0.0, 0.0, 0.0};
  double dbacc = 0.0;
  bool odd = false;   // PM_SPLIT3: dA negated in this stage

  // piece q of an operand: row piece q % NRP, column group q / NRP
  auto gload = [&](uint4 (*buf)[RPP], int64_t k0) {
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int piece = tid + i * NTH;
      const bool isA = piece < PA;
      const int q = isA ? piece : piece - PA;
      const int rp = q % NRP, cg = q / NRP;
      const int col = (isA ? n0 : j0) + cg * EPP;
      const int lim = isA ? N : J;
      // rows past the split range load a clamped row (zeroed when stored to
      // LDS); columns past the end only reach outputs that are never stored
      const int colc = col < lim ? col : lim - EPP;
#pragma unroll
      for (int u = 0; u < RPP; ++u) {
        const int64_t row = k0 + rp * RPP + u;
        const int64_t rowc = row < r1 ? row : r1 - 1;
        buf[i][u] = isA ? *(const uint4*)(A + rowc * lda + colc) : *(const uint4*)(B + rowc * ldh + colc);
      }
    }
    __builtin_amdgcn_sched_barrier(0);   // keep the prefetch where it is issued
  };
  auto lstore = [&](const uint4 (*buf)[RPP], int stage, int64_t k0) {
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int piece = tid + i * NTH;
      if (piece >= PIECES) continue;
      const bool isA = piece < PA;
      const int q = isA ? piece : piece - PA;
      const int rp = q % NRP, cg = q / NRP;
      char* base = lds + stage * STAGE + (isA ? 0 : REGA);
      const uint32_t m0k = (k0 + rp * RPP < r1) ? 0xffffffffu : 0u;            // row validity masks
      const uint32_t m1k = (k0 + rp * RPP + RPP - 1 < r1) ? 0xffffffffu : 0u;
      if constexpr (SPL) {
        // rows 2 rp and 2 rp + 1: one word of high pieces, one of low pieces
        const float* x0 = (const float*)&buf[i][0];
        const float* x1 = (const float*)&buf[i][RPP - 1];
#pragma unroll
        for (int e = 0; e < EPP; ++e) {
          const bf16 h0 = (bf16)x0[e], h1 = (bf16)x1[e];
          const bf16 l0 = (bf16)(x0[e] - (float)h0), l1 = (bf16)(x1[e] - (float)h1);
          char* line = base + dw_col(cg * EPP + e) + rp * 4;
          *(uint32_t*)line = ((uint32_t)__builtin_bit_cast(uint16_t, h0) & m0k & 0xffffu) |
                             (((uint32_t)__builtin_bit_cast(uint16_t, h1) << 16) & m1k);
          *(uint32_t*)(line + 32) = ((uint32_t)__builtin_bit_cast(uint16_t, l0) & m0k & 0xffffu) |
                                    (((uint32_t)__builtin_bit_cast(uint16_t, l1) << 16) & m1k);
        }
      } else if (ES == 2) {
        const uint16_t* lo = (const uint16_t*)&buf[i][0];
        const uint16_t* hi = (const uint16_t*)&buf[i][RPP - 1];
#pragma unroll
        for (int e = 0; e < EPP; ++e)
          *(uint32_t*)(base + dw_col(cg * EPP + e) + rp * 4) =
              ((uint32_t)lo[e] & m0k & 0xffffu) | (((uint32_t)hi[e] << 16) & m1k);
      } else {
        const uint32_t* v = (const uint32_t*)&buf[i][0];
#pragma unroll
        for (int e = 0; e < EPP; ++e) *(uint32_t*)(base + dw_col(cg * EPP + e) + rp * 4) = v[e] & m0k;
      }
    }
  };
  auto compute = [&](int stage, int64_t k0) {
    const char* base = lds + stage * STAGE;
    if constexpr (PM == PM_F64) {
      // fp32 rows of each column line, four at a time through the fp64 product
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int ro = (4 * kk + (lane >> 4)) * 4;
        double av[2], bv[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          av[h] = (double)*(const float*)(base + dw_col(32 * wm + 16 * h + (lane & 15)) + ro);
          bv[h] = (double)*(const float*)(base + REGA + dw_col(32 * wn + 16 * h + (lane & 15)) + ro);
        }
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int b = 0; b < 2; ++b) accd[a][b] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[a], bv[b], accd[a][b], 0, 0, 0);
      }
    }
    if constexpr (SPL) {
      // high pieces at byte 0 of a column line, low pieces at byte 32
      const int koff = (lane >> 5) * 16;
      bf16x8 ap[NT][2], bp[NT][2];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          ap[t][c] = *(const bf16x8*)(base + dw_col(32 * (wm * NT + t) + (lane & 31)) + 32 * c + koff);
          bp[t][c] = *(const bf16x8*)(base + REGA + dw_col(32 * (wn * NT + t) + (lane & 31)) + 32 * c + koff);
        }
#pragma unroll
      for (int a = 0; a < NT; ++a)
#pragma unroll
        for (int b = 0; b < NT; ++b) mma_split<2>(acc[a][b], ap[a], bp[b]);
    }
#pragma unroll
    for (int c = 0; c < (PM == PM_F64 || SPL ? 0 : NCH); ++c) {
      const int koff = c * 32 + (lane >> 5) * (8 * ES);
      frag af[NT], bf[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        af[t] = *(const frag*)(base + dw_col(32 * (wm * NT + t) + (lane & 31)) + koff);
        bf[t] = *(const frag*)(base + REGA + dw_col(32 * (wn * NT + t) + (lane & 31)) + koff);
      }
      if constexpr (PM != PM_NATIVE) {
        // PM_SPLIT3 negates dA on every other stage and subtracts those
        // stages in the fp64 fold (the matrix core's one-signed bias cancels)
        constexpr int NP = PM == PM_SPLIT3 ? 3 : 2;
        bf16x8 ap[NT][NP], bp[NT][NP];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          split_frag<NP>(PM == PM_SPLIT3 && odd ? -af[t] : af[t], ap[t]);
          split_frag<NP>(bf[t], bp[t]);
        }
#pragma unroll
        for (int a = 0; a < NT; ++a)
#pragma unroll
          for (int b = 0; b < NT; ++b) mma_split<NP>(acc[a][b], ap[a], bp[b]);
      } else {
#pragma unroll
        for (int a = 0; a < NT; ++a)
#pragma unroll
          for (int b = 0; b < NT; ++b) Elem<T>::mma(acc[a][b], af[a], bf[b]);
      }
    }
    if constexpr (PM == PM_SPLIT3) {
#pragma unroll
      for (int a = 0; a < NT; ++a)
#pragma unroll
        for (int b = 0; b < NT; ++b)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            acc64[a][b][r] += odd ? -(double)acc[a][b][r] : (double)acc[a][b][r];
            acc[a][b][r] = 0.0f;
          }
      odd = !odd;
    }
    // bias cotangent: value rows of this slice, one column per thread
    // (the 64-byte column line is read as 16 independent words)
    if (pdb && tj == 0 && tid < BNn && k0 < rv) {
      const int nr = (int)((rv - k0) < SR ? (rv - k0) : SR);
      const uint32_t* colw = (const uint32_t*)(base + dw_col(tid));
      typename std::conditional<ES == 4, double, float>::type part_sum = 0;
#pragma unroll
      for (int w = 0; w < 16; ++w) {
        const uint32_t v = colw[w];
        if constexpr (SPL) {
          // words 0-7: high pieces of rows 2w, 2w + 1; words 8-15: low pieces
          if (w < 8) {
            const uint32_t l = colw[w + 8];
            const double r0 = (double)(float)__builtin_bit_cast(bf16, (uint16_t)(v & 0xffffu)) +
                              (double)(float)__builtin_bit_cast(bf16, (uint16_t)(l & 0xffffu));
            const double r1 = (double)(float)__builtin_bit_cast(bf16, (uint16_t)(v >> 16)) +
                              (double)(float)__builtin_bit_cast(bf16, (uint16_t)(l >> 16));
            part_sum += (2 * w < nr ? r0 : 0.0) + (2 * w + 1 < nr ? r1 : 0.0);
          }
        } else if constexpr (ES == 2) {
          const float lo = Elem<T>::to_f(__builtin_bit_cast(T, (uint16_t)(v & 0xffffu)));
          const float hi = Elem<T>::to_f(__builtin_bit_cast(T, (uint16_t)(v >> 16)));
          part_sum += (2 * w < nr ? lo : 0.0f) + (2 * w + 1 < nr ? hi : 0.0f);
        } else {
          part_sum += w < nr ? (double)__uint_as_float(v) : 0.0;
        }
      }
      dbacc += (double)part_sum;
    }
  };

  if constexpr (OCC >= 2 || NB > 2) {
    // two LDS stages and a ring of NB register buffers: buffer b holds the
    // stages s = b (mod NB), so NB stages of loads are in flight while one is
    // multiplied.  Loads are unconditional (stage index clamped, rows past
    // the range zeroed at the LDS store), so the waits are static counts.
    uint4 bufs[NB][PPT][RPP];
    const int last = nst > 0 ? nst - 1 : 0;
#pragma unroll
    for (int b = 0; b < NB; ++b) gload(bufs[b], r0 + (int64_t)(b < last ? b : last) * SR);
    if (nst > 0) lstore(bufs[0], 0, r0);
    gload(bufs[0], r0 + (int64_t)(NB < last ? NB : last) * SR);
    lds_sync();
    for (int st = 0; st < nst; st += NB) {
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        const int sc = st + u;                     // stage in LDS[sc & 1]
        if (sc >= nst) break;
        compute(sc & 1, r0 + (int64_t)sc * SR);
        __builtin_amdgcn_sched_barrier(0);
        if (sc + 1 < nst) lstore(bufs[(u + 1) % NB], (sc + 1) & 1, r0 + (int64_t)(sc + 1) * SR);
        gload(bufs[(u + 1) % NB], r0 + (int64_t)(sc + 1 + NB < last ? sc + 1 + NB : last) * SR);
        lds_sync();
      }
    }
  } else {
    // large tiles (one wave per SIMD): one register buffer, one stage ahead
    uint4 b0[PPT][RPP];
    if (nst > 0) {
      gload(b0, r0);
      lstore(b0, 0, r0);
    }
    lds_sync();
    for (int st = 0; st < nst; ++st) {
      gload(b0, r0 + (int64_t)(st + 1 < nst ? st + 1 : st) * SR);
      compute(st & 1, r0 + (int64_t)st * SR);
      __builtin_amdgcn_sched_barrier(0);
      if (st + 1 < nst) lstore(b0, (st + 1) & 1, r0 + (int64_t)(st + 1) * SR);
      lds_sync();
    }
  }

  const int hh = lane >> 5;
  const int64_t obase = ((int64_t)g * n_split + split) * (int64_t)N * J;
  if constexpr (PM == PM_F64) {
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int j = j0 + 32 * wn + 16 * b + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int n = n0 + 32 * wm + 16 * a + (lane >> 4) + 4 * r;
          if (n < N && j < J) partial64[obase + (int64_t)n * J + j] = accd[a][b][r];
        }
      }
  }
#pragma unroll
  for (int a = 0; a < (PM == PM_F64 ? 0 : NT); ++a) {
#pragma unroll
    for (int b = 0; b < NT; ++b) {
      const int j = j0 + 32 * (wn * NT + b) + (lane & 31);
      if (j >= J) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int n = n0 + 32 * (wm * NT + a) + 8 * (r >> 2) + 4 * hh + (r & 3);
        if (n >= N) continue;
        if constexpr (A64) partial64[obase + (int64_t)n * J + j] = acc64[a][b][r];
        else partial[obase + (int64_t)n * J + j] = acc[a][b][r];
      }
    }
  }
  if (pdb && tj == 0 && tid < BNn && n0 + tid < N)
    pdb[((int64_t)g * n_split + split) * N + n0 + tid] = dbacc;
}

// ---------------------------------------------------------------------------
// k_gemm_dw_tr: the same weight gradient for 16-bit storage, with row-major
// operand stages in LDS.  Global loads are whole 16-byte row segments, 16
// lanes per 256-byte row (fully used cache lines); the matrix-core fragments,
// which need 8 consecutive rows of one column per lane, are gathered with the
// transposing LDS read of gfx950: within each 16-lane group, lanes 4r..4r+3
// address the four 8-byte pieces of row r of a 4 x 16 block and lane i
// receives column i of the block.  Two such reads give a lane its 8 rows.
// Row pitch = row bytes + pad with pitch/4 = 16 or 48 (mod 64), so the four
// rows of one read fall in disjoint bank ranges.
// ---------------------------------------------------------------------------
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 tr_bf16x4;
typedef __attribute__((__vector_size__(4 * sizeof(__fp16)))) __fp16 tr_f16x4;

template <class T>
__device__ __forceinline__ u32x2 lds_read_tr(const char* p) {
  if constexpr (__is_same(T, bf16)) {
    return __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                                         (__attribute__((address_space(3))) tr_bf16x4*)(p)));
  } else {
    return __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4f16(
                                         (__attribute__((address_space(3))) tr_f16x4*)(p)));
  }
}

// The same transposing read issued as an instruction the compiler does not
// model.  Stages filled by LDS DMA (global_load_lds) are guarded by explicit
// vmcnt waits and barriers; with the intrinsic, the compiler cannot tell the
// DMA targets apart from the stage being read and drains every DMA in flight
// (vmcnt(0)) before each stage's reads, which leaves nothing prefetched.  The
// caller waits for these reads itself (lgkm_wait below).
__device__ __forceinline__ u32x2 lds_read_tr_raw(const char* p) {
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
  u32x2 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r) : "v"(a));
  return r;
}

// s_waitcnt lgkmcnt(N) that the values read before it flow through, so no
// use of them is scheduled ahead of the wait
template <int N, int K>
__device__ __forceinline__ void lgkm_wait(u32x4 (&v)[K]) {
  static_assert(N >= 0 && N <= 15, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
#pragma unroll
  for (int i = 0; i < K; ++i) asm volatile("" : "+v"(v[i]));
}

__host__ __device__ constexpr int dw_tr_pitch(int row_bytes) {
  // smallest pitch >= row_bytes (multiple of 64 bytes) with pitch/4 = 16 or 48 mod 64
  return (row_bytes / 4) % 64 == 16 || (row_bytes / 4) % 64 == 48 ? row_bytes
         : (row_bytes / 4) % 64 == 0 ? row_bytes + 64 : row_bytes + 64 * ((row_bytes / 4) % 64 == 32 ? 1 : 0);
}

// NS > 0 (tile sides of 128 or 256 columns): the stages move straight from
// global memory into an NS-deep LDS ring (global_load_lds_dwordx4).  Rows are
// then unpadded (256 or 512 bytes); the 16-byte segment s of row r sits at
// s ^ 4 (r & 3), which keeps the four rows of a transposing read in disjoint
// bank ranges.
template <class T, int WM, int WN, int NT, int NB, int NS = 0, int OCC = 2>
__global__ void __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu(OCC)))
k_gemm_dw_tr(const T* __restrict__ dA, int64_t a_g, int64_t lda, const T* __restrict__ H, int64_t h_g,
             int64_t ldh, int64_t R, int64_t n_value, int N, int J, float* __restrict__ partial,
             double* __restrict__ pdb, int n_split, int64_t rows_per_split) {
  static_assert(sizeof(T) == 2, "16-bit storage only");
  constexpr int BNn = 32 * NT * WM;
  constexpr int BJ = 32 * NT * WN;
  constexpr int NTH = 64 * WM * WN;
  constexpr int SR = 32;                    // rows per stage (two 16-row k chunks)
  constexpr int SA = BNn / 8, SB = BJ / 8;  // 16-byte segments per row
  constexpr int PA = dw_tr_pitch(BNn * 2), PB = dw_tr_pitch(BJ * 2);
  constexpr int REGA = SR * PA;
  constexpr int STAGE = REGA + SR * PB;
  constexpr int PIECES = SR * (SA + SB);
  static_assert(PIECES % NTH == 0, "whole pieces per thread");
  constexpr int PPT = PIECES / NTH;
  static_assert(NS == 0 || ((BNn == 128 || BNn == 256) && (BJ == 128 || BJ == 256) && NS >= 2),
                "direct-to-LDS stages: tile sides of 128 or 256");
  constexpr int RBA = BNn * 2, RBB = BJ * 2;  // unpadded ring row bytes
  constexpr int DSTAGE = SR * (RBA + RBB);    // ring stage: SR rows of A, then SR rows of B
  constexpr int LDSB = NS > 0 ? NS * DSTAGE : 2 * STAGE;
  typedef typename Elem<T>::frag frag;
  __shared__ __attribute__((aligned(16))) char lds[LDSB];

  const int tiles_n = (N + BNn - 1) / BNn;
  const int tiles = tiles_n * ((J + BJ - 1) / BJ);
  const int64_t lb = xcd_remap(blockIdx.x, gridDim.x);
  const int tile = (int)(lb % tiles);
  const int tn = tile % tiles_n;
  const int tj = tile / tiles_n;
  const int split = (int)(lb / tiles);
  const int g = blockIdx.z;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % WM;
  const int wn = wave / WM;
  const int n0 = tn * BNn;
  const int j0 = tj * BJ;
  // stages are dealt round-robin over the splits (split s takes stages s,
  // s + n_split, ...), so at any time the blocks stream one contiguous window
  // of rows (page and DRAM locality) instead of n_split separate ranges
  (void)rows_per_split;
  const int64_t r1 = R;
  const int64_t rv = R < n_value ? R : n_value;
  const int64_t tot = (R + SR - 1) / SR;
  const int nst = (int)(split < tot ? (tot - split + n_split - 1) / n_split : 0);
  auto krow = [&](int sc) { return ((int64_t)split + (int64_t)sc * n_split) * SR; };
  const T* A = dA + g * a_g;
  const T* B = H + g * h_g;

  f32x16 acc[NT][NT];
#pragma unroll
  for (int a = 0; a < NT; ++a)
#pragma unroll
    for (int b = 0; b < NT; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;
  float dbp[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) dbp[t] = 0.0f;
  double dbacc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) dbacc[t] = 0.0;
  const bool want_db = pdb && tj == 0 && wn == 0;

  // piece q: operand A for q < SR * SA (row q / SA, segment q % SA), else B.
  // Rows past the range load a clamped row and are zeroed at the LDS store;
  // columns past the end load a clamped column (never stored outputs).
  auto gload = [&](u32x4* buf, int64_t k0) {
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int q = tid + i * NTH;
      const bool isA = q < SR * SA;
      const int qq = isA ? q : q - SR * SA;
      const int sg = isA ? qq % SA : qq % SB;
      const int row = isA ? qq / SA : qq / SB;
      int64_t gr = k0 + row;
      if (gr >= r1) gr = r1 - 1;
      int col = (isA ? n0 : j0) + sg * 8;
      const int lim = isA ? N : J;
      if (col >= lim) col = lim - 8;
      buf[i] = isA ? *(const u32x4*)(A + gr * lda + col) : *(const u32x4*)(B + gr * ldh + col);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  auto lstore = [&](const u32x4* buf, int stage, int64_t k0) {
    char* base = lds + stage * STAGE;
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int q = tid + i * NTH;
      const bool isA = q < SR * SA;
      const int qq = isA ? q : q - SR * SA;
      const int sg = isA ? qq % SA : qq % SB;
      const int row = isA ? qq / SA : qq / SB;
      const uint32_t m = (k0 + row < r1) ? 0xffffffffu : 0u;
      const u32x4 v = buf[i] & m;
      *(u32x4*)(base + (isA ? row * PA : REGA + row * PB) + sg * 16) = v;
    }
  };
  // fragments: lane l holds rows 8 (l / 32) .. +7 of its column (l % 32) of
  // the 32-column block, as two transposing reads of 4 rows
  const int grp = lane >> 4, t16 = lane & 15;
  const int rr = t16 >> 2, qq4 = t16 & 3;
  const int kb = 8 * (lane >> 5);
  auto frag_at = [&](const char* region, int pitch, int c, int colblk) {
    const int byte = (colblk + 16 * (grp & 1) + 4 * qq4) * 2;
    // the row of both reads is = rr (mod 4): one swizzle for the pair
    const char* p0 = NS > 0 ? region + (c * 16 + kb + rr) * pitch + (((byte >> 4) ^ (4 * rr)) << 4) + (byte & 15)
                            : region + (c * 16 + kb + rr) * pitch + byte;
    const u32x2 lo = lds_read_tr<T>(p0);
    const u32x2 hi = lds_read_tr<T>(p0 + 4 * pitch);
    const u32x4 w = {lo.x, lo.y, hi.x, hi.y};
    return __builtin_bit_cast(frag, w);
  };
  // DMA stages: raw transposing reads of the fragments.  Four-wave blocks
  // read both 16-row chunks up front and start the first chunk's products
  // once its reads have landed; larger blocks (which would lose occupancy to
  // the extra registers) read one chunk at a time.
  auto frag_raw = [&](const char* region, int pitch, int c, int colblk) {
    const int byte = (colblk + 16 * (grp & 1) + 4 * qq4) * 2;
    const char* p0 = region + (c * 16 + kb + rr) * pitch + (((byte >> 4) ^ (4 * rr)) << 4) + (byte & 15);
    const u32x2 lo = lds_read_tr_raw(p0);
    const u32x2 hi = lds_read_tr_raw(p0 + 4 * pitch);
    return u32x4{lo.x, lo.y, hi.x, hi.y};
  };
  auto compute_dma = [&](int stage, int64_t k0) {
    static_assert(SR == 32, "two 16-row chunks per stage");
    const char* base = lds + stage * DSTAGE;
    const char* bbase = base + SR * RBA;
    constexpr bool AHEAD = NTH <= 256;
    u32x4 w[2][2 * NT];   // chunk c: A fragments 0..NT-1, then B fragments
    auto read_chunk = [&](int c) {
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        w[c][t] = frag_raw(base, RBA, c, 32 * (wm * NT + t));
        w[c][NT + t] = frag_raw(bbase, RBB, c, 32 * (wn * NT + t));
      }
    };
    read_chunk(0);
    if constexpr (AHEAD) read_chunk(1);
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      if (c == 1 && !AHEAD) read_chunk(1);
      if (c == 0 && AHEAD) lgkm_wait<4 * NT>(w[0]);   // the second chunk's 4 NT reads may still be in flight
      else lgkm_wait<0>(w[c]);
      frag af[NT], bf[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        af[t] = __builtin_bit_cast(frag, w[c][t]);
        bf[t] = __builtin_bit_cast(frag, w[c][NT + t]);
      }
      // the stages hold clamped copies of the last row past R: their dA
      // elements (rows k0 + 16 c + kb + e of this lane) contribute zero
      if (k0 + SR > r1) {
        const int64_t rw0 = k0 + c * 16 + kb;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (rw0 + e >= r1) af[t][e] = Elem<T>::from_f(0.0f);
      }
#pragma unroll
      for (int a = 0; a < NT; ++a)
#pragma unroll
        for (int b = 0; b < NT; ++b) Elem<T>::mma(acc[a][b], af[a], bf[b]);
      if (want_db && k0 + c * 16 < rv) {
        const int64_t rw0 = k0 + c * 16 + kb;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int e = 0; e < 8; ++e) dbp[t] += rw0 + e < rv ? Elem<T>::to_f(af[t][e]) : 0.0f;
      }
    }
    if (want_db) {
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        dbacc[t] += (double)dbp[t];
        dbp[t] = 0.0f;
      }
    }
  };
  auto compute = [&](int stage, int64_t k0) {
    const char* base = lds + stage * (NS > 0 ? DSTAGE : STAGE);
    const char* bbase = base + (NS > 0 ? SR * RBA : REGA);
#pragma unroll
    for (int c = 0; c < SR / 16; ++c) {
      frag af[NT], bf[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        af[t] = frag_at(base, NS > 0 ? RBA : PA, c, 32 * (wm * NT + t));
        bf[t] = frag_at(bbase, NS > 0 ? RBB : PB, c, 32 * (wn * NT + t));
      }
#pragma unroll
      for (int a = 0; a < NT; ++a)
#pragma unroll
        for (int b = 0; b < NT; ++b) Elem<T>::mma(acc[a][b], af[a], bf[b]);
      // bias cotangent: value rows of the lane's 8 rows of its dA columns
      if (want_db && k0 + c * 16 < rv) {
        const int64_t rw0 = k0 + c * 16 + kb;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
          for (int e = 0; e < 8; ++e) dbp[t] += rw0 + e < rv ? Elem<T>::to_f(af[t][e]) : 0.0f;
      }
    }
    if (want_db) {
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        dbacc[t] += (double)dbp[t];
        dbp[t] = 0.0f;
      }
    }
  };

  if constexpr (NS > 0) {
    // One DMA instruction of a wave fills 1 KB: 1024 / RB rows of one
    // operand (RB = its row bytes), lane l at byte 16 l (physical segment
    // l % (RB / 16) of its row, holding the logical segment of that index
    // ^ 4 (row & 3)).  A stage is GA such groups of A rows and GB of B rows,
    // dealt to the waves round-robin.  Rows past R (in the last stage, at
    // most) load a clamped row; compute() zeroes their dA elements.  Every
    // stage is a DMA stage, so the waits below are the only ones on the
    // ring (a register-loaded stage made the compiler drain every load in
    // flight before each stage's LDS reads).
    constexpr int GA = SR * RBA / 1024, GB = SR * RBB / 1024;
    constexpr int NG = GA + GB;
    constexpr int NW = NTH / 64;
    static_assert(NG % NW == 0, "whole row groups per wave");
    constexpr int GPW = NG / NW;
    static_assert((NS - 2) * GPW <= 63, "outstanding loads exceed the vmcnt range");
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const T* dsrc[GPW];
    int64_t dld[GPW];
    int drow[GPW];
#pragma unroll
    for (int i = 0; i < GPW; ++i) {
      const int gq = wv + i * NW;
      const bool isA = gq < GA;
      const int spr = (isA ? RBA : RBB) / 16;  // segments per row
      const int row = (isA ? gq : gq - GA) * (64 / spr) + lane / spr;
      const int sg = (lane % spr) ^ (4 * (row & 3));
      int col = (isA ? n0 : j0) + sg * 8;
      const int lim = isA ? N : J;
      if (col >= lim) col = lim - 8;
      dsrc[i] = (isA ? A : B) + col;
      dld[i] = isA ? lda : ldh;
      drow[i] = row;
    }
    auto issue = [&](int sc, int buf) {
      const int64_t k0 = krow(sc);
      char* dst = lds + buf * DSTAGE;
#pragma unroll
      for (int i = 0; i < GPW; ++i) {
        int64_t gr = k0 + drow[i];
        if (gr > r1 - 1) gr = r1 - 1;
        __builtin_amdgcn_global_load_lds((const void*)(dsrc[i] + gr * dld[i]),
                                         (lds_ptr_t)(dst + (wv + i * NW) * 1024), 16, 0, 0);
      }
    };
#pragma unroll
    for (int b = 0; b < NS - 1; ++b)
      if (b < nst) issue(b, b);
    int stg = 0;
    for (int sc = 0; sc < nst; ++sc) {
      const int later = nst - 1 - sc;
      if constexpr (NS >= 4) {
        if (later >= 2) wait_vmcnt<2 * GPW>();
        else if (later == 1) wait_vmcnt<GPW>();
        else wait_vmcnt<0>();
      } else if constexpr (NS == 3) {
        if (later >= 1) wait_vmcnt<GPW>();
        else wait_vmcnt<0>();
      } else {
        wait_vmcnt<0>();
      }
      lds_sync();
      if (sc + NS - 1 < nst) issue(sc + NS - 1, stg == 0 ? NS - 1 : stg - 1);
      compute_dma(stg, krow(sc));
      stg = stg + 1 == NS ? 0 : stg + 1;
    }
  } else {
  // ring of NB register stages (as in k_gemm_dw)
  u32x4 bufs[NB][PPT];
  const int last = nst > 0 ? nst - 1 : 0;
#pragma unroll
  for (int b = 0; b < NB; ++b) gload(bufs[b], krow(b < last ? b : last));
  if (nst > 0) lstore(bufs[0], 0, krow(0));
  gload(bufs[0], krow(NB < last ? NB : last));
  lds_sync();
  for (int st = 0; st < nst; st += NB) {
#pragma unroll
    for (int u = 0; u < NB; ++u) {
      const int sc = st + u;
      if (sc >= nst) break;
      compute(sc & 1, krow(sc));
      __builtin_amdgcn_sched_barrier(0);
      if (sc + 1 < nst) lstore(bufs[(u + 1) % NB], (sc + 1) & 1, krow(sc + 1));
      gload(bufs[(u + 1) % NB], krow(sc + 1 + NB < last ? sc + 1 + NB : last));
      lds_sync();
    }
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
  if (want_db) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      double v = dbacc[t];
      v += __shfl_xor(v, 32);                      // the other 8-row half of the same column
      const int n = n0 + 32 * (wm * NT + t) + (lane & 31);
      if (lane < 32 && n < N) pdb[((int64_t)g * n_split + split) * N + n] = v;
    }
  }
}

// ---------------------------------------------------------------------------
// host launchers
// ---------------------------------------------------------------------------
namespace {

// Tiles.  A wave owns 32 points x 32*NT columns of every stream.  Layers
// below the wide path: NT = 4 / 2 / 1 for 1 / 2 / 3+ streams (2 x 2 waves,
// two waves per SIMD), and 4 x 1 waves for narrow layers (N <= 32).  The wide
// path (K, N >= 256) stages operands straight into an LDS ring, which
// hides the load latency that otherwise bounds it, and uses the block shapes
// measured fastest per stream count.
}  // namespace

bool nt_resident_ok(int elem_bytes, int C, int K, int N, int64_t n_points, int64_t ldx, int64_t ldo) {
  const int64_t span = (n_points + 1) * (ldx > ldo ? ldx : ldo) * (int64_t)elem_bytes;
  return elem_bytes == 2 && C >= 1 && C <= 5 && K == 128 && N == 128 && span < ((int64_t)1 << 31);
}

namespace {

// compute units of the current device (cached per device)
int cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev] <= 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

template <class T, int C>
constexpr bool wide_ok() { return sizeof(T) == 2 && (C == 1 || C == 3 || C == 5); }

template <class T, int ND1, int ND2, int EPI>
hipError_t nt_dispatch_tile(const NtArgs<T>& a, int G, hipStream_t st) {
  constexpr int C = 1 + ND1 + ND2;
  constexpr int NTM = C == 1 ? 4 : (C == 2 ? 2 : 1);
  const int64_t npts = a.seg.n_points;
  if (npts <= 0) return hipSuccess;
  if ((a.pm != PM_NATIVE && sizeof(T) != 4) || (a.kx > 0 && (sizeof(T) != 2 || a.K != 2 * a.kx)))
    return hipErrorInvalidValue;
  if constexpr (sizeof(T) == 4) {
    // split products (the critic and the generators' sensor rows): one or two
    // streams; register-staged tiles
    if (a.pm != PM_NATIVE) {
      if (a.y || a.fp1) return hipErrorInvalidValue;
      if constexpr (C <= 2) {
        if (a.N <= 32 && a.pm != PM_F64) {
          dim3 grid((unsigned)(((npts + 127) / 128) * ((a.N + 31) / 32)), 1, G);
          if (a.pm == PM_SPLIT2) k_gemm_nt<T, ND1, ND2, 4, 1, 1, 1, EPI, 2, true, 0, PM_SPLIT2><<<grid, 256, 0, st>>>(a);
          else k_gemm_nt<T, ND1, ND2, 4, 1, 1, 1, EPI, 2, true, 0, PM_SPLIT3><<<grid, 256, 0, st>>>(a);
        } else if (a.pm == PM_SPLIT2 && C == 1 && a.N >= 256 && npts >= 16384) {
          // 128 points x 256 columns, 4 x 4 waves of 1 x 2 fragments, a ring
          // of 3 register stages (the fastest measured for the sensor rows
          // at K = N = 1024)
          if constexpr (C == 1) {
            dim3 grid((unsigned)(((npts + 127) / 128) * ((a.N + 255) / 256)), 1, G);
            k_gemm_nt<T, ND1, ND2, 4, 4, 1, 2, EPI, 1, true, 0, PM_SPLIT2, 3><<<grid, 1024, 0, st>>>(a);
          }
        } else if (a.pm == PM_SPLIT2 && C == 1 && a.N <= 128) {
          // 64 points x 128 columns, 2 x 2 waves (no idle column half at N = 128)
          if constexpr (C == 1) {
            dim3 grid((unsigned)(((npts + 63) / 64) * ((a.N + 127) / 128)), 1, G);
            k_gemm_nt<T, ND1, ND2, 2, 2, 1, 2, EPI, 2, true, 0, PM_SPLIT2><<<grid, 256, 0, st>>>(a);
          }
        } else if (a.pm == PM_SPLIT2) {
          // 64 points x 64 NTM columns, 2 x 2 waves
          constexpr int BN = 64 * NTM;
          dim3 grid((unsigned)(((npts + 63) / 64) * ((a.N + BN - 1) / BN)), 1, G);
          k_gemm_nt<T, ND1, ND2, 2, 2, 1, NTM, EPI, 2, true, 0, PM_SPLIT2><<<grid, 256, 0, st>>>(a);
        } else if (a.pm == PM_F64) {
          // fp64 products: 64 x 64 tiles
          dim3 grid((unsigned)(((npts + 63) / 64) * ((a.N + 63) / 64)), 1, G);
          k_gemm_nt<T, ND1, ND2, 2, 2, 1, 1, EPI, 2, true, 0, PM_F64><<<grid, 256, 0, st>>>(a);
        } else {
          // fp64 stage sums: 64 x 64 tiles
          dim3 grid((unsigned)(((npts + 63) / 64) * ((a.N + 63) / 64)), 1, G);
          k_gemm_nt<T, ND1, ND2, 2, 2, 1, 1, EPI, 2, true, 0, PM_SPLIT3><<<grid, 256, 0, st>>>(a);
        }
        return hipGetLastError();
      } else {
        return hipErrorInvalidValue;
      }
    }
  }
  if constexpr (sizeof(T) == 2 && C <= 5 && EPI != EPI_DF) {
    const bool skip = a.skip || a.skip_g || a.out_gh;
    const bool two = a.kx > 0;   // two-term weight rows: the operand is kx wide
    if (nt_resident_ok((int)sizeof(T), C, two ? a.kx : a.K, a.N, npts, a.ldx, a.ldo) &&
        !(skip && (a.fp1 || a.y)) && (!two || (EPI == EPI_FWD && a.K == 2 * a.kx))) {
      // persistent weight-resident kernel: two blocks per CU in total (one
      // for the five-stream skip variant)
      const int64_t ntiles = (npts + 31) / 32;
      // one-stream launches (sensor rows: few tiles, small blocks) take three
      // blocks per CU
      int64_t nb = (skip || (two && C >= 5) ? wr_blocks_per_cu<C, true>() : (C == 1 ? 3 : 2)) * (int64_t)cu_count() / G;
      if (nb < 1) nb = 1;
      if (nb > ntiles) nb = ntiles;
      dim3 grid((unsigned)nb, 1, G);
      if constexpr (EPI == EPI_FWD) {
        if (two) {
          if (a.fp1) k_gemm_nt_wr<T, ND1, ND2, EPI, true, false, true><<<grid, 256, 0, st>>>(a, ntiles);
          else if (skip) k_gemm_nt_wr<T, ND1, ND2, EPI, false, true, true><<<grid, 256, 0, st>>>(a, ntiles);
          else k_gemm_nt_wr<T, ND1, ND2, EPI, false, false, true><<<grid, 256, 0, st>>>(a, ntiles);
          return hipGetLastError();
        }
      }
      if (a.fp1) k_gemm_nt_wr<T, ND1, ND2, EPI, true><<<grid, 256, 0, st>>>(a, ntiles);
      else if (skip) k_gemm_nt_wr<T, ND1, ND2, EPI, false, true><<<grid, 256, 0, st>>>(a, ntiles);
      else k_gemm_nt_wr<T, ND1, ND2, EPI, false><<<grid, 256, 0, st>>>(a, ntiles);
      return hipGetLastError();
    }
  }
  if (a.y || a.fp1) return hipErrorInvalidValue;  // output / first-layer fusion only in the resident kernel
  if constexpr (EPI == EPI_DF) {
    if (a.skip || a.skip_g || a.out_gh) return hipErrorInvalidValue;
  }
  if (a.N <= 32) {
    dim3 grid((unsigned)(((npts + 127) / 128) * ((a.N + 31) / 32)), 1, G);
    k_gemm_nt<T, ND1, ND2, 4, 1, 1, 1, EPI, (C >= 4 ? 1 : 2)><<<grid, 256, 0, st>>>(a);
  } else if (wide_ok<T, C>() && a.K >= 256 && a.N >= 256) {
    // wide layers: operand stages loaded straight into an LDS ring several
    // stages ahead, larger wave tiles (fewer LDS fragment reads per MFMA) and
    // fewer L2 re-reads of each activation tile.  Tile shapes are the
    // fastest measured per stream count, epilogue and depth (K = 256 layers
    // are bound by HBM traffic, K >= 512 by the matrix cores).
    const bool deep = a.K >= 512;
    if constexpr (!wide_ok<T, C>()) {
      return hipErrorInvalidValue;
    } else if constexpr (C == 1) {
      if constexpr (EPI == EPI_BWD) {
        if (deep) {
          // 128 points x 256 columns, 2 x 4 fragments per wave, 3-stage ring
          dim3 grid((unsigned)(((npts + 127) / 128) * ((a.N + 255) / 256)), 1, G);
          k_gemm_nt<T, ND1, ND2, 2, 2, 2, 4, EPI, 2, true, 3><<<grid, 256, 0, st>>>(a);
          return hipGetLastError();
        }
      }
      if (((npts + 127) / 128) * ((a.N + 127) / 128) * G < 64) {
        // short launches (a critic's batch): 32 points x 128 columns, four
        // waves of one fragment, for four times the blocks
        dim3 grid((unsigned)(((npts + 31) / 32) * ((a.N + 127) / 128)), 1, G);
        k_gemm_nt<T, ND1, ND2, 1, 4, 1, 1, EPI, 2, true, 3><<<grid, 256, 0, st>>>(a);
      } else {
        // 128 points x 128 columns, 2 x 2 fragments per wave, 3-stage ring
        dim3 grid((unsigned)(((npts + 127) / 128) * ((a.N + 127) / 128)), 1, G);
        k_gemm_nt<T, ND1, ND2, 2, 2, 2, 2, EPI, 2, true, 3><<<grid, 256, 0, st>>>(a);
      }
    } else if constexpr ((C == 5 || C == 3) && EPI == EPI_BWD) {
      if constexpr (C == 3) {
        if (deep) {
          // eight waves (2 x 4), 64 points x 256 columns, 3-stage ring
          dim3 grid((unsigned)(((npts + 63) / 64) * ((a.N + 255) / 256)), 1, G);
          k_gemm_nt<T, ND1, ND2, 2, 4, 1, 2, EPI, 1, false, 3><<<grid, 512, 0, st>>>(a);
          return hipGetLastError();
        }
      }
      // four waves (1 x 4), 32 points x 128 columns, 3-stage ring: two blocks
      // per CU, so that one block's epilogue (the jet carry, VALU work a third
      // to three quarters as long as its products) runs beside the other's
      // products (five streams: 8-10 % faster than eight waves of 32 x 256 or
      // 64 x 128 at K = 1024 and 256; three streams at K = 256: 15 % faster
      // than the register-staged 64 x 128 tile)
      dim3 grid((unsigned)(((npts + 31) / 32) * ((a.N + 127) / 128)), 1, G);
      k_gemm_nt<T, ND1, ND2, 1, 4, 1, 1, EPI, 2, true, 3><<<grid, 256, 0, st>>>(a);
    } else {
      if constexpr (C == 3 && EPI == EPI_FWD) {
        if (!deep) {
          // eight waves (2 x 4), 64 points x 128 columns, 4-stage ring
          dim3 grid((unsigned)(((npts + 63) / 64) * ((a.N + 127) / 128)), 1, G);
          k_gemm_nt<T, ND1, ND2, 2, 4, 1, 1, EPI, 2, true, 4><<<grid, 512, 0, st>>>(a);
          return hipGetLastError();
        }
      }
      // eight waves (2 x 4), 64 points x 256 columns, 3-stage ring (6-11 %
      // faster than 4 stages at K = 1024, two-term forward and reverse)
      dim3 grid((unsigned)(((npts + 63) / 64) * ((a.N + 255) / 256)), 1, G);
      k_gemm_nt<T, ND1, ND2, 2, 4, 1, 2, EPI, 1, false, 3><<<grid, 512, 0, st>>>(a);
    }
  } else {
    constexpr int BN = 64 * NTM;
    dim3 grid((unsigned)(((npts + 63) / 64) * ((a.N + BN - 1) / BN)), 1, G);
    k_gemm_nt<T, ND1, ND2, 2, 2, 1, NTM, EPI, (C >= 7 ? 1 : 2)><<<grid, 256, 0, st>>>(a);
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
  // 16-bit storage, both sides >= 512: 256 x 256 tiles of 16 waves, about
  // 256 blocks (one per CU; as fast as 512 and half the partials to write and
  // reduce); otherwise about 1024 blocks of the 128 x 128 (or smaller) tile
  // grid, and 512 for a single output tile (each split writes a whole N x J
  // fp32 partial, and one resident wave of blocks suffices)
  const bool big = elem_bytes == 2 && N >= 512 && J >= 512;
  const int bt = big ? 256 : (N >= 128 && J >= 128) ? 128 : ((N >= 64 && J >= 64) ? 64 : 32);
  const int64_t tiles = (int64_t)((N + bt - 1) / bt) * ((J + bt - 1) / bt) * G;
  const int64_t target = big ? 256 : (tiles == 1 ? 512 : 1024);
  int64_t want = (target + tiles - 1) / tiles;
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
                          int n_split, int64_t rows_per_split, int G, hipStream_t st, int pm, double* partial64) {
  if (R <= 0) return hipSuccess;
  if (pm != PM_NATIVE && sizeof(T) != 4) return hipErrorInvalidValue;
  if ((pm == PM_SPLIT3 || pm == PM_F64) && !partial64) return hipErrorInvalidValue;
  if constexpr (sizeof(T) == 4) {
    if (pm == PM_F64) {
      dim3 grid((unsigned)(((N + 63) / 64) * ((J + 63) / 64)) * n_split, 1, G);
      k_gemm_dw<T, 2, 2, 1, 2, 2, PM_F64><<<grid, 256, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, J, partial,
                                                              pdb, n_split, rows_per_split, partial64);
      return hipGetLastError();
    }
    if (pm != PM_NATIVE) {
#define PIGAN_DW_PM(WM_, WN_, NT_, NTH_, BT_)                                                                     \
  do {                                                                                                           \
    dim3 grid((unsigned)(((N + BT_ - 1) / BT_) * ((J + BT_ - 1) / BT_)) * n_split, 1, G);                         \
    if (pm == PM_SPLIT2)                                                                                         \
      k_gemm_dw<T, WM_, WN_, NT_, 2, 4, PM_SPLIT2><<<grid, NTH_, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, \
                                                                       J, partial, pdb, n_split, rows_per_split,   \
                                                                       partial64);                                 \
    else                                                                                                         \
      k_gemm_dw<T, WM_, WN_, NT_, 2, 2, PM_SPLIT3><<<grid, NTH_, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, \
                                                                       J, partial, pdb, n_split, rows_per_split,   \
                                                                       partial64);                                 \
  } while (0)
      if (N >= 256 && J >= 256 && pm == PM_SPLIT2) {
        // 256 x 256, 16 waves of 64 x 64 (the fastest measured at 1024 x 1024)
        dim3 grid((unsigned)(((N + 255) / 256) * ((J + 255) / 256)) * n_split, 1, G);
        k_gemm_dw<T, 4, 4, 2, 1, 2, PM_SPLIT2><<<grid, 1024, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, J,
                                                                     partial, pdb, n_split, rows_per_split,
                                                                     partial64);
      } else if (N >= 128 && J >= 128) PIGAN_DW_PM(2, 2, 2, 256, 128);
      else if (N >= 64 && J >= 64) PIGAN_DW_PM(2, 2, 1, 256, 64);
      else PIGAN_DW_PM(1, 1, 1, 64, 32);
#undef PIGAN_DW_PM
      return hipGetLastError();
    }
  }
  if constexpr (sizeof(T) == 2) {
    // operand stages straight into an LDS ring; 64 x 64 columns per wave.
    // Block shapes per width are the fastest measured.
    if (N >= 512 && J >= 512) {
      // 256 x 256, 16 waves, 2-stage ring
      dim3 grid((unsigned)(((N + 255) / 256) * ((J + 255) / 256)) * n_split, 1, G);
      k_gemm_dw_tr<T, 4, 4, 2, 4, 2, 1><<<grid, 1024, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, J, partial,
                                                              pdb, n_split, rows_per_split);
    } else if (N >= 128 && J >= 256) {
      // 128 x 256, 8 waves, 3-stage ring
      dim3 grid((unsigned)(((N + 127) / 128) * ((J + 255) / 256)) * n_split, 1, G);
      k_gemm_dw_tr<T, 2, 4, 2, 4, 3, 1><<<grid, 512, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, J, partial,
                                                             pdb, n_split, rows_per_split);
    } else if (N >= 128 && J >= 128) {
      // 128 x 128, 4 waves, 3-stage ring
      dim3 grid((unsigned)(((N + 127) / 128) * ((J + 127) / 128)) * n_split, 1, G);
      k_gemm_dw_tr<T, 2, 2, 2, 4, 3><<<grid, 256, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, J, partial, pdb,
                                                          n_split, rows_per_split);
    } else if (N >= 64 && J >= 64) {
      dim3 grid((unsigned)(((N + 63) / 64) * ((J + 63) / 64)) * n_split, 1, G);
      k_gemm_dw_tr<T, 2, 2, 1, 4><<<grid, 256, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, J, partial, pdb,
                                                       n_split, rows_per_split);
    } else {
      dim3 grid((unsigned)(((N + 31) / 32) * ((J + 31) / 32)) * n_split, 1, G);
      k_gemm_dw_tr<T, 1, 1, 1, 4><<<grid, 64, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, J, partial, pdb,
                                                      n_split, rows_per_split);
    }
    return hipGetLastError();
  }
  if (N >= 128 && J >= 128) {
    dim3 grid((unsigned)(((N + 127) / 128) * ((J + 127) / 128)) * n_split, 1, G);
    k_gemm_dw<T, 2, 2, 2, 2, 4><<<grid, 256, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, J, partial, pdb,
                                                    n_split, rows_per_split, nullptr);
  } else if (N >= 64 && J >= 64) {
    dim3 grid((unsigned)(((N + 63) / 64) * ((J + 63) / 64)) * n_split, 1, G);
    k_gemm_dw<T, 2, 2, 1, 2, 4><<<grid, 256, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, J, partial, pdb,
                                                 n_split, rows_per_split, nullptr);
  } else {
    dim3 grid((unsigned)(((N + 31) / 32) * ((J + 31) / 32)) * n_split, 1, G);
    k_gemm_dw<T, 1, 1, 1, 2, 4><<<grid, 64, 0, st>>>(dA, a_g, lda, H, h_g, ldh, R, n_value, N, J, partial, pdb,
                                                n_split, rows_per_split, nullptr);
  }
  return hipGetLastError();
}

#define PIGAN_INST(T)                                                                                    \
  template hipError_t launch_gemm_nt<T>(int, int, int, const NtArgs<T>&, int, hipStream_t);              \
  template hipError_t launch_gemm_dw<T>(const T*, int64_t, int64_t, const T*, int64_t, int64_t, int64_t, \
                                        int64_t, int, int, float*, double*, int, int64_t, int, hipStream_t, int, \
                                        double*);
PIGAN_INST(float)
PIGAN_INST(bf16)
PIGAN_INST(f16)
#undef PIGAN_INST

}  // namespace pigan
