// K-means++ seeding in the kernel's feature space: D^2 sampling of the
// centers among the points (Arthur and Vassilvitskii), the initialization
// the paper cites for its convergence properties (Section II-B) and leaves
// to future work (Section V).
//
// With centers c_0 .. c_{t-1} chosen, D(i) = min_s ||phi(x_i) - phi(x_cs)||^2
// where ||phi(x) - phi(y)||^2 = K(x,x) - 2 K(x,y) + K(y,y) (the kernel trick
// of Section II-B).  Center t is the first index i with P(i) > u_t * S
// (P the prefix sums of D in index order, S = P(n-1)), so i is drawn with
// probability D(i)/S; the uniforms u_t come from the caller.
//
// The entries of K are computed from the staged points, whatever the K
// storage mode, and the three entries of a distance by the same routine, so
// a point that coincides with a center has distance exactly 0.  One pass per
// center (16 lanes per point, so each group reads its row in 256-byte runs)
// updates D, each point's nearest center (lowest position on ties) and
// per-block fp64 sums of D; a single workgroup then walks the prefix sums to
// the drawn index.  Everything stays on the device: the host only
// enqueues the 2k - 1 launches.
#include "tile_mma.h"

#include <climits>

namespace kkm {

namespace {

constexpr int kSeedThr = 256;               // threads per workgroup
constexpr int kSeedLanes = 16;              // lanes per point
constexpr int kSeedPts = kSeedThr / kSeedLanes;  // points per workgroup (one block of D)

// The dot product x_i . x_c (or, for the Gaussian, |x_i - x_c|^2) over a
// row of d_pad floats, by a group of 16 lanes: lane l takes the 16-byte
// chunks l, l + 16, ... in order, then a fixed shuffle tree adds the lanes.
// The split depends on the column only, so identical rows give identical sums.
template <int KIND>
__device__ inline float group_sum(const float* __restrict__ xi, const float* __restrict__ xc, int d4, int l) {
  float s = 0.f;
  for (int c = l; c < d4; c += kSeedLanes) {
    const float4 a = ((const float4*)xi)[c], b = ((const float4*)xc)[c];
    if (KIND == GAUSS) {
      float t = a.x - b.x;
      s = fmaf(t, t, s);
      t = a.y - b.y;
      s = fmaf(t, t, s);
      t = a.z - b.z;
      s = fmaf(t, t, s);
      t = a.w - b.w;
      s = fmaf(t, t, s);
    } else {
      s = fmaf(a.x, b.x, s);
      s = fmaf(a.y, b.y, s);
      s = fmaf(a.z, b.z, s);
      s = fmaf(a.w, b.w, s);
    }
  }
#pragma unroll
  for (int off = kSeedLanes / 2; off > 0; off >>= 1) s += __shfl_xor(s, off, kSeedLanes);
  return s;
}

// kappa from the group sum: the Gaussian takes the squared difference.
template <int KIND>
__device__ inline float kentry(float s, const KappaParams& kp) {
  if (KIND == GAUSS) return __builtin_amdgcn_exp2f(kp.neg_g_log2e * s);
  return kappa<KIND>(s, 0.f, 0.f, kp);
}

// Pass for center t (its index is c_first when t = 0, else centers[t]).
// kd[i] = K(i,i) by the same routine (written when t = 0).  V, when not
// null, receives each point's nearest center (the last pass).  Block b of D
// is the kSeedPts points of workgroup b; bsum[b] their fp64 sum (fixed tree).
template <int KIND>
__global__ __launch_bounds__(kSeedThr) void kpp_dist_kernel(const float* __restrict__ Xp, int64_t n, int d_pad,
                                                           KappaParams kp, int* __restrict__ centers, int t,
                                                           int c_first, float* __restrict__ kd,
                                                           float* __restrict__ D, float* __restrict__ best,
                                                           int* __restrict__ bestc, double* __restrict__ bsum,
                                                           int* __restrict__ V) {
  __shared__ double red[kSeedPts];
  const int tid = threadIdx.x, l = tid % kSeedLanes, p = tid / kSeedLanes;
  const int64_t i = (int64_t)blockIdx.x * kSeedPts + p;
  const int c = t == 0 ? c_first : centers[t];
  if (t == 0 && blockIdx.x == 0 && tid == 0) centers[0] = c_first;
  const int d4 = d_pad / 4;
  const float* xc = Xp + (int64_t)c * d_pad;
  const float* xi = Xp + (i < n ? i : c) * d_pad;  // rows past n read the center's (unused)
  const float kic = kentry<KIND>(group_sum<KIND>(xi, xc, d4, l), kp);
  float kii, kcc;
  if (t == 0) {
    kii = KIND == GAUSS ? 1.f : kentry<KIND>(group_sum<KIND>(xi, xi, d4, l), kp);
    kcc = KIND == GAUSS ? 1.f : kentry<KIND>(group_sum<KIND>(xc, xc, d4, l), kp);
  }
  float dv = 0.f;
  if (i < n && l == 0) {
    if (t == 0) {
      kd[i] = kii;
    } else {
      kii = kd[i];
      kcc = kd[c];
    }
    const float d2 = i == c ? 0.f : fmaxf((kii + kcc) - 2.f * kic, 0.f);
    float bd = d2;
    int bc = t;
    if (t > 0) {
      const float b0 = best[i];
      if (!(d2 < b0)) {
        bd = b0;
        bc = bestc[i];
      }
    }
    best[i] = bd;
    bestc[i] = bc;
    dv = t == 0 ? d2 : fminf(D[i], d2);
    D[i] = dv;
    if (V) V[i] = bc;
  }
  if (l == 0) red[p] = (double)dv;
  __syncthreads();
  for (int w = kSeedPts / 2; w > 0; w >>= 1) {
    if (tid < w) red[tid] += red[tid + w];
    __syncthreads();
  }
  if (tid == 0) bsum[blockIdx.x] = red[0];
}

// Inclusive prefix sums of v over the workgroup's threads (fixed tree,
// Hillis-Steele over kSeedThr entries); buf holds 2 x kSeedThr doubles.
__device__ inline double block_scan(double v, double* buf) {
  const int tid = threadIdx.x;
  int cur = 0;
  buf[tid] = v;
  __syncthreads();
  for (int off = 1; off < kSeedThr; off <<= 1) {
    buf[(cur ^ 1) * kSeedThr + tid] = buf[cur * kSeedThr + tid] + (tid >= off ? buf[cur * kSeedThr + tid - off] : 0.0);
    cur ^= 1;
    __syncthreads();
  }
  const double r = buf[cur * kSeedThr + tid];
  __syncthreads();
  return r;
}

// The lowest index not among centers[0 .. t-1] (one thread).
__device__ inline int lowest_unused(const int* __restrict__ centers, int t, int64_t n) {
  for (int64_t i = 0; i < n; ++i) {
    bool used = false;
    for (int s2 = 0; s2 < t; ++s2) used |= (centers[s2] == (int)i);
    if (!used) return (int)i;
  }
  return -1;
}

// Draws center t from D with the uniform ut: the first index whose prefix
// sum exceeds ut * S, with D(i) > 0.  Three levels, each prefix-summed in
// parallel by a fixed tree: runs of block sums (one per thread), the blocks
// of the run holding the target, the points of the block holding it; at each
// level the lowest qualifying entry wins.  The levels' sums are associated
// differently, so rounding can leave a level short of the target: then its
// last entry with a positive weight is taken.  If S = 0, the lowest index not
// yet chosen.
__global__ __launch_bounds__(kSeedThr) void kpp_select_kernel(const float* __restrict__ D, const double* __restrict__ bsum,
                                                             int nblk, int64_t n, double ut,
                                                             int* __restrict__ centers, int t) {
  __shared__ double buf[2 * kSeedThr];
  __shared__ int s_vote;
  __shared__ double s_val;
  const int tid = threadIdx.x;
  // lowest (or highest) thread whose flag is set, -1 if none; all threads call
  auto vote = [&](bool q, bool lowest) {
    if (tid == 0) s_vote = lowest ? INT_MAX : -1;
    __syncthreads();
    if (q) {
      if (lowest) atomicMin(&s_vote, tid);
      else atomicMax(&s_vote, tid);
    }
    __syncthreads();
    const int f = s_vote;
    __syncthreads();
    return f == INT_MAX ? -1 : f;
  };
  auto bcast = [&](double v, int src) {
    if (tid == src) s_val = v;
    __syncthreads();
    const double r = s_val;
    __syncthreads();
    return r;
  };

  // level 1: runs of `per` block sums, one per thread, added in order
  const int per = (nblk + kSeedThr - 1) / kSeedThr;
  const int b0 = tid * per, b1 = min(nblk, b0 + per);
  double r = 0.0;
  for (int b = b0; b < b1; b += 8) {  // eight loads in flight
    double v[8];
#pragma unroll
    for (int x = 0; x < 8; ++x) v[x] = bsum[min(b + x, nblk - 1)];
#pragma unroll
    for (int x = 0; x < 8; ++x)
      if (b + x < b1) r += v[x];
  }
  const double P1 = block_scan(r, buf);
  const double S = bcast(P1, kSeedThr - 1);
  if (!(S > 0.0)) {
    if (tid == 0) centers[t] = lowest_unused(centers, t, n);
    return;
  }
  const double target = ut * S;
  int j = vote(r > 0.0 && P1 > target, true);
  if (j < 0) j = vote(r > 0.0, false);
  double base = bcast(P1 - r, j);

  // level 2: the blocks of run j, kSeedThr at a time
  const int m_lo = j * per, m_hi = min(nblk, m_lo + per);
  int blk = -1, fb_blk = -1;
  double fb_base = 0.0;
  for (int m0 = m_lo; m0 < m_hi && blk < 0; m0 += kSeedThr) {
    const int m = m0 + tid;
    const double v = m < m_hi ? bsum[m] : 0.0;
    const double P2 = base + block_scan(v, buf);
    const int f = vote(v > 0.0 && P2 > target, true);
    if (f >= 0) {
      blk = m0 + f;
      base = bcast(P2 - v, f);
    } else {
      const int lp = vote(v > 0.0, false);
      if (lp >= 0) {
        fb_blk = m0 + lp;
        fb_base = bcast(P2 - v, lp);
      }
      base = bcast(P2, kSeedThr - 1);
    }
  }
  if (blk < 0) {
    blk = fb_blk;
    base = fb_base;
  }

  // level 3: the points of block blk
  const int64_t i0 = (int64_t)blk * kSeedPts;
  const float x = (tid < kSeedPts && i0 + tid < n) ? D[i0 + tid] : 0.f;
  const double P3 = base + block_scan((double)x, buf);
  int f = vote(x > 0.f && P3 > target, true);
  if (f < 0) f = vote(x > 0.f, false);
  if (tid == 0) centers[t] = f >= 0 ? (int)(i0 + f) : lowest_unused(centers, t, n);
}

}  // namespace

int seed_blocks(int64_t n) { return (int)((n + kSeedPts - 1) / kSeedPts); }

hipError_t launch_kpp_dist(const float* Xp, int64_t n, int d_pad, const KappaParams& kp, int* centers, int t,
                           int c_first, float* kd, float* D, float* best, int* bestc, double* bsum, int* V,
                           hipStream_t s) {
  const dim3 grid((unsigned)seed_blocks(n)), block(kSeedThr);
  switch (kp.kind) {
    case LINEAR:
      hipLaunchKernelGGL(kpp_dist_kernel<LINEAR>, grid, block, 0, s, Xp, n, d_pad, kp, centers, t, c_first, kd, D,
                         best, bestc, bsum, V);
      break;
    case POLY:
      hipLaunchKernelGGL(kpp_dist_kernel<POLY>, grid, block, 0, s, Xp, n, d_pad, kp, centers, t, c_first, kd, D,
                         best, bestc, bsum, V);
      break;
    default:
      hipLaunchKernelGGL(kpp_dist_kernel<GAUSS>, grid, block, 0, s, Xp, n, d_pad, kp, centers, t, c_first, kd, D,
                         best, bestc, bsum, V);
      break;
  }
  return hipGetLastError();
}

hipError_t launch_kpp_select(const float* D, const double* bsum, int64_t n, double ut, int* centers, int t,
                             hipStream_t s) {
  hipLaunchKernelGGL(kpp_select_kernel, dim3(1), dim3(kSeedThr), 0, s, D, bsum, seed_blocks(n), n, ut, centers, t);
  return hipGetLastError();
}

}  // namespace kkm
