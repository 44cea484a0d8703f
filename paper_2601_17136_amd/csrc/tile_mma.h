// Device building blocks shared by the K-build and on-the-fly kernels: the
// fp32 MFMA mainloop of one 128 x 128 tile of B = X X^T, and the kernel
// functions kappa applied to its entries.
#pragma once
#include "kkm_internal.h"

namespace kkm {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kLdsK = kBK + 4;              // padded k stride: conflict-free 16-byte reads
constexpr int kLdsBuf = 2 * kTile * kLdsK;  // one stage: A and B chunk
constexpr int kLdsFloats = 2 * kLdsBuf;     // double-buffered: 40 KB

// acc[bi][bj][r] = sum_k Xa[i][k] Xb[j][k] for the 128 x 128 tile whose rows
// start at Xa and columns at Xb (row stride d_pad, d_pad a multiple of 8):
//   i = wm*64 + bi*32 + 8*(r/4) + 4*h + r%4,   j = wn*64 + bj*32 + lane%32
// with wave = 2*wm + wn and h = lane/32.  256 threads; ends with a barrier, so
// the caller may reuse lds right away.
//
// Within a 16-wide k chunk the half-wave h takes k = 8h .. 8h+7 and step s of
// v_mfma_f32_32x32x2_f32 pairs k = s with k = 8 + s: every lane fetches its
// operands with two 16-byte LDS reads per 32-row block.  When d_pad is an odd
// multiple of 8 the last chunk is 8 wide: its upper half is neither loaded
// nor multiplied (h takes k = 4h .. 4h+3, four steps), so a row pays for at
// most 7 zero columns.
__device__ inline void mma_tile(const float* __restrict__ Xa, const float* __restrict__ Xb,
                                int d_pad, float* lds, floatx16 acc[2][2]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l32 = lane & 31, h = lane >> 5;
  const int f0 = tid, f1 = tid + 256;
  const float* Ag0 = Xa + (int64_t)(f0 >> 2) * d_pad + (f0 & 3) * 4;
  const float* Ag1 = Xa + (int64_t)(f1 >> 2) * d_pad + (f1 & 3) * 4;
  const float* Bg0 = Xb + (int64_t)(f0 >> 2) * d_pad + (f0 & 3) * 4;
  const float* Bg1 = Xb + (int64_t)(f1 >> 2) * d_pad + (f1 & 3) * 4;
  const int so0 = (f0 >> 2) * kLdsK + (f0 & 3) * 4;
  const int so1 = (f1 >> 2) * kLdsK + (f1 & 3) * 4;
  const int nkf = d_pad / kBK;                  // full 16-wide chunks
  const bool half_last = (d_pad % kBK) != 0;    // then one 8-wide chunk
  const int nk = nkf + (half_last ? 1 : 0);
  // in the 8-wide chunk, the threads at k offsets 8 and 12 load nothing
  // (f1 = f0 + 256 has the same k offset as f0)
  const bool upper = (f0 & 3) >= 2;
  const float4 zero4 = {0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[bi][bj][r] = 0.f;

  const bool skip0 = nkf == 0 && upper;
  float4 ra0 = skip0 ? zero4 : *(const float4*)Ag0, ra1 = skip0 ? zero4 : *(const float4*)Ag1;
  float4 rb0 = skip0 ? zero4 : *(const float4*)Bg0, rb1 = skip0 ? zero4 : *(const float4*)Bg1;
  *(float4*)(lds + so0) = ra0;
  *(float4*)(lds + so1) = ra1;
  *(float4*)(lds + kTile * kLdsK + so0) = rb0;
  *(float4*)(lds + kTile * kLdsK + so1) = rb1;
  __syncthreads();

  for (int kc = 0; kc < nkf; ++kc) {
    const int cur = kc & 1;
    if (kc + 1 < nk) {  // prefetch the next chunk into registers
      const int ko = (kc + 1) * kBK;
      const bool skip = kc + 1 == nkf && upper;  // the next chunk is the 8-wide one
      ra0 = skip ? zero4 : *(const float4*)(Ag0 + ko);
      ra1 = skip ? zero4 : *(const float4*)(Ag1 + ko);
      rb0 = skip ? zero4 : *(const float4*)(Bg0 + ko);
      rb1 = skip ? zero4 : *(const float4*)(Bg1 + ko);
    }
    const float* As = lds + cur * kLdsBuf;
    const float* Bs = As + kTile * kLdsK;
    float a[2][8], bv[2][8];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const float* pa = As + (wm * 64 + q * 32 + l32) * kLdsK + h * 8;
      const float* pb = Bs + (wn * 64 + q * 32 + l32) * kLdsK + h * 8;
      const float4 a0 = *(const float4*)pa, a1 = *(const float4*)(pa + 4);
      const float4 b0 = *(const float4*)pb, b1 = *(const float4*)(pb + 4);
      a[q][0] = a0.x; a[q][1] = a0.y; a[q][2] = a0.z; a[q][3] = a0.w;
      a[q][4] = a1.x; a[q][5] = a1.y; a[q][6] = a1.z; a[q][7] = a1.w;
      bv[q][0] = b0.x; bv[q][1] = b0.y; bv[q][2] = b0.z; bv[q][3] = b0.w;
      bv[q][4] = b1.x; bv[q][5] = b1.y; bv[q][6] = b1.z; bv[q][7] = b1.w;
    }
#pragma unroll
    for (int s = 0; s < 8; ++s)
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[bi][s], bv[bj][s], acc[bi][bj], 0, 0, 0);
    if (kc + 1 < nk) {
      float* nxt = lds + (cur ^ 1) * kLdsBuf;
      *(float4*)(nxt + so0) = ra0;
      *(float4*)(nxt + so1) = ra1;
      *(float4*)(nxt + kTile * kLdsK + so0) = rb0;
      *(float4*)(nxt + kTile * kLdsK + so1) = rb1;
    }
    __syncthreads();
  }
  if (half_last) {  // the 8-wide chunk, in buffer nkf & 1: h takes k = 4h .. 4h+3
    const float* As = lds + (nkf & 1) * kLdsBuf;
    const float* Bs = As + kTile * kLdsK;
    float a[2][4], bv[2][4];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const float4 a0 = *(const float4*)(As + (wm * 64 + q * 32 + l32) * kLdsK + h * 4);
      const float4 b0 = *(const float4*)(Bs + (wn * 64 + q * 32 + l32) * kLdsK + h * 4);
      a[q][0] = a0.x; a[q][1] = a0.y; a[q][2] = a0.z; a[q][3] = a0.w;
      bv[q][0] = b0.x; bv[q][1] = b0.y; bv[q][2] = b0.z; bv[q][3] = b0.w;
    }
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[bi][s], bv[bj][s], acc[bi][bj], 0, 0, 0);
    __syncthreads();
  }
}

// ---- Small widths (d_pad <= kRegMaxDpad): the sweep kernels' product.
// A workgroup stages its block's 128 rows in LDS once (stride 2 HP + 4
// floats); each wavefront (wm, wn) loads its 64 columns of the current tile
// into registers: lane (l, h) holds column l of each 32-column block at
// k = h*HP .. h*HP + HP - 1 (HP = d_pad / 2), and step s of
// v_mfma_f32_32x32x2_f32 pairs k = s with k = HP + s.
constexpr int kRegMaxDpad = 64;

template <int HP>
__device__ inline void load_operand(const float* __restrict__ Y, int64_t row, int d_pad, int h, float (&v)[HP]) {
  const float4* p = (const float4*)(Y + row * d_pad + h * HP);
#pragma unroll
  for (int u = 0; u < HP / 4; ++u) {
    const float4 t = p[u];
    v[4 * u] = t.x;
    v[4 * u + 1] = t.y;
    v[4 * u + 2] = t.z;
    v[4 * u + 3] = t.w;
  }
}

// acc[bi][bj] for one bj: the wavefront's 64 rows from As (stride 2 HP + 4
// floats, an odd number of 16-byte units, so the 16-byte reads of 32
// consecutive rows are conflict-free) against its 32 columns bj in b.  The
// two column blocks run as two passes, so the second block's loads are still
// in flight while the first block's products run.
template <int HP>
__device__ inline void mma_rows_lds(const float* __restrict__ As, const float (&b)[HP], floatx16& acc0,
                                    floatx16& acc1, int l32, int h) {
  constexpr int ldsA = 2 * HP + 4;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    acc0[r] = 0.f;
    acc1[r] = 0.f;
  }
  const float* p0 = As + l32 * ldsA + h * HP;
  const float* p1 = p0 + 32 * ldsA;
  // rows of the next four steps read one group ahead; the scheduling
  // barriers keep the reads from being hoisted further (registers)
  float4 a0 = *(const float4*)p0, a1 = *(const float4*)p1;
#pragma unroll
  for (int s4 = 0; s4 < HP; s4 += 4) {
    float4 n0 = a0, n1 = a1;
    if (s4 + 4 < HP) {
      n0 = *(const float4*)(p0 + s4 + 4);
      n1 = *(const float4*)(p1 + s4 + 4);
    }
    const float av0[4] = {a0.x, a0.y, a0.z, a0.w}, av1[4] = {a1.x, a1.y, a1.z, a1.w};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(av0[u], b[s4 + u], acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(av1[u], b[s4 + u], acc1, 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    a0 = n0;
    a1 = n1;
  }
}

// kappa(x, y) from b = x.y (and the squared norms nx, ny for the Gaussian):
//   LINEAR b;  POLY (gamma b + c)^degree;  GAUSS exp(-gamma (nx + ny - 2b)).
template <int KIND>
__device__ inline float kappa(float b, float nx, float ny, const KappaParams& kp) {
  if (KIND == LINEAR) return b;
  if (KIND == POLY) {
    float t = fmaf(kp.gamma, b, kp.coef0), v = 1.f;
    for (int e = kp.degree; e > 0; e >>= 1) {  // t^degree by squaring
      if (e & 1) v *= t;
      t *= t;
    }
    return v;
  }
  const float s = fmaxf(nx + ny - 2.f * b, 0.f);
  return __builtin_amdgcn_exp2f(kp.neg_g_log2e * s);
}

// Whether a Gaussian entry formed by the expansion may be off by more than
// the tolerance: gamma * err(s) * K with err(s) ~ 8 * 2^-24 * (nx + ny).
__device__ inline bool gauss_needs_fix(float v, float nx, float ny, const KappaParams& kp) {
  return kp.fix_scale * (nx + ny) * v > kp.fix_tol;
}

// The Gaussian entry from b = x.y and u = c(|x|^2 + |y|^2), c = -gamma log2(e)
// (the norms scaled once per row and column): exp2(c s) with
// c s = -2c b + u, clamped at 0 (s >= 0).  Two operations fewer per entry
// than kappa<GAUSS> with its estimate below, for the same value up to
// rounding.
__device__ inline float gauss_scaled(float b, float u, const KappaParams& kp) {
  return __builtin_amdgcn_exp2f(fminf(fmaf(kp.m2c, b, u), 0.f));
}

// gauss_needs_fix in the scaled form: fix_scale (|x|^2 + |y|^2) v > fix_tol,
// multiplied through by c < 0.
__device__ inline bool gauss_needs_fix_scaled(float v, float u, const KappaParams& kp) {
  return u * v < kp.fix_uthr;
}

// The Gaussian entry from the coordinate differences (fp32, d_pad terms).
__device__ inline float gauss_direct(const float* __restrict__ x, const float* __restrict__ y,
                                     int d_pad, const KappaParams& kp) {
  float s = 0.f;
  for (int c = 0; c < d_pad; c += 4) {
    const float4 a = *(const float4*)(x + c), b = *(const float4*)(y + c);
    float t = a.x - b.x;
    s = fmaf(t, t, s);
    t = a.y - b.y;
    s = fmaf(t, t, s);
    t = a.z - b.z;
    s = fmaf(t, t, s);
    t = a.w - b.w;
    s = fmaf(t, t, s);
  }
  return __builtin_amdgcn_exp2f(kp.neg_g_log2e * s);
}

}  // namespace kkm
