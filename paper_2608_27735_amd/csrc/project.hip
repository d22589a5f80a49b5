// project.hip -- EWA projection of 3D Gaussians (forward) and its chain rule
// (backward), one thread per Gaussian.
//
// The paper renders the active partition with 3D Gaussian Splatting
// (Introduction; Method section). Each Gaussian is projected to a 2D Gaussian:
// mean by the pinhole map, covariance by the first-order (EWA) approximation
// J W Sigma W^T J^T of the perspective map, dilated by eps2d, colour from real
// spherical harmonics of the view direction, opacity by a sigmoid.
//
// The values that decide culling, the tile rectangle and the depth key are
// computed with a fixed fp32 operation order (no contraction, correctly
// rounded division and square root, exp of the log-scale taken in double and
// rounded once), so binning is reproducible bit for bit on any IEEE machine
// that follows the same order.
#include "abcd_internal.h"

namespace abcd {
namespace {

// Real orthonormal spherical harmonics to degree 3 of a unit direction, index
// l^2 + l + m, written as homogeneous harmonic polynomials:
//   l=1: y, z, x;  l=2: xy, yz, 2z^2-x^2-y^2, xz, x^2-y^2;
//   l=3: y(3x^2-y^2), xyz, y(4z^2-x^2-y^2), z(2z^2-3x^2-3y^2),
//        x(4z^2-x^2-y^2), z(x^2-y^2), x(x^2-3y^2),
// each with its normalisation constant.
constexpr float kY0 = 0.28209479177387814f;   // 1/(2 sqrt(pi))
constexpr float kY1 = 0.48860251190291992f;   // sqrt(3/(4 pi))
constexpr float kY2a = 1.0925484305920792f;   // sqrt(15/pi)/2
constexpr float kY2b = 0.31539156525252005f;  // sqrt(5/pi)/4
constexpr float kY2c = 0.54627421529603959f;  // sqrt(15/pi)/4
constexpr float kY3a = 0.59004358992664352f;  // sqrt(35/(2 pi))/4
constexpr float kY3b = 2.8906114426405538f;   // sqrt(105/pi)/2
constexpr float kY3c = 0.45704579946446572f;  // sqrt(21/(2 pi))/4
constexpr float kY3d = 0.37317633259011540f;  // sqrt(7/pi)/4
constexpr float kY3e = 1.4453057213202769f;   // sqrt(105/pi)/4

// Y[16] and, when G != nullptr, dY/d(x, y, z) as G[16][3].
__device__ __forceinline__ void sh_eval(int degree, float x, float y, float z, float* Y, float* G) {
  Y[0] = kY0;
  if (G) G[0] = G[1] = G[2] = 0.0f;
  if (degree < 1) return;
  Y[1] = kY1 * y;
  Y[2] = kY1 * z;
  Y[3] = kY1 * x;
  if (G) {
    G[3] = 0; G[4] = kY1; G[5] = 0;
    G[6] = 0; G[7] = 0; G[8] = kY1;
    G[9] = kY1; G[10] = 0; G[11] = 0;
  }
  if (degree < 2) return;
  const float xx = x * x, yy = y * y, zz = z * z;
  Y[4] = kY2a * x * y;
  Y[5] = kY2a * y * z;
  Y[6] = kY2b * (2.0f * zz - xx - yy);
  Y[7] = kY2a * x * z;
  Y[8] = kY2c * (xx - yy);
  if (G) {
    G[12] = kY2a * y; G[13] = kY2a * x; G[14] = 0;
    G[15] = 0; G[16] = kY2a * z; G[17] = kY2a * y;
    G[18] = -2.0f * kY2b * x; G[19] = -2.0f * kY2b * y; G[20] = 4.0f * kY2b * z;
    G[21] = kY2a * z; G[22] = 0; G[23] = kY2a * x;
    G[24] = 2.0f * kY2c * x; G[25] = -2.0f * kY2c * y; G[26] = 0;
  }
  if (degree < 3) return;
  Y[9] = kY3a * y * (3.0f * xx - yy);
  Y[10] = kY3b * x * y * z;
  Y[11] = kY3c * y * (4.0f * zz - xx - yy);
  Y[12] = kY3d * z * (2.0f * zz - 3.0f * xx - 3.0f * yy);
  Y[13] = kY3c * x * (4.0f * zz - xx - yy);
  Y[14] = kY3e * z * (xx - yy);
  Y[15] = kY3a * x * (xx - 3.0f * yy);
  if (G) {
    G[27] = kY3a * 6.0f * x * y; G[28] = kY3a * 3.0f * (xx - yy); G[29] = 0;
    G[30] = kY3b * y * z; G[31] = kY3b * x * z; G[32] = kY3b * x * y;
    G[33] = -2.0f * kY3c * x * y; G[34] = kY3c * (4.0f * zz - xx - 3.0f * yy);
    G[35] = 8.0f * kY3c * y * z;
    G[36] = -6.0f * kY3d * x * z; G[37] = -6.0f * kY3d * y * z;
    G[38] = kY3d * (6.0f * zz - 3.0f * xx - 3.0f * yy);
    G[39] = kY3c * (4.0f * zz - 3.0f * xx - yy); G[40] = -2.0f * kY3c * x * y;
    G[41] = 8.0f * kY3c * x * z;
    G[42] = 2.0f * kY3e * x * z; G[43] = -2.0f * kY3e * y * z; G[44] = kY3e * (xx - yy);
    G[45] = kY3a * 3.0f * (xx - yy); G[46] = -6.0f * kY3a * x * y; G[47] = 0;
  }
}

// sum_b w[b] dY_b/d(x, y, z): the SH gradient contracted with per-basis
// weights, without materialising the 16 x 3 table.
template <int D>
__device__ __forceinline__ void sh_grad_dot(float x, float y, float z, const float* w, float* g) {
  g[0] = g[1] = g[2] = 0.0f;
  if (D < 1) return;
  g[0] += kY1 * w[3];
  g[1] += kY1 * w[1];
  g[2] += kY1 * w[2];
  if (D < 2) return;
  const float xx = x * x, yy = y * y, zz = z * z;
  g[0] += kY2a * (y * w[4] + z * w[7]) - 2.0f * kY2b * x * w[6] + 2.0f * kY2c * x * w[8];
  g[1] += kY2a * (x * w[4] + z * w[5]) - 2.0f * kY2b * y * w[6] - 2.0f * kY2c * y * w[8];
  g[2] += kY2a * (y * w[5] + x * w[7]) + 4.0f * kY2b * z * w[6];
  if (D < 3) return;
  g[0] += kY3a * 6.0f * x * y * w[9] + kY3b * y * z * w[10] - 2.0f * kY3c * x * y * w[11] -
          6.0f * kY3d * x * z * w[12] + kY3c * (4.0f * zz - 3.0f * xx - yy) * w[13] +
          2.0f * kY3e * x * z * w[14] + kY3a * 3.0f * (xx - yy) * w[15];
  g[1] += kY3a * 3.0f * (xx - yy) * w[9] + kY3b * x * z * w[10] +
          kY3c * (4.0f * zz - xx - 3.0f * yy) * w[11] - 6.0f * kY3d * y * z * w[12] -
          2.0f * kY3c * x * y * w[13] - 2.0f * kY3e * y * z * w[14] - 6.0f * kY3a * x * y * w[15];
  g[2] += kY3b * x * y * w[10] + 8.0f * kY3c * y * z * w[11] +
          kY3d * (6.0f * zz - 3.0f * xx - 3.0f * yy) * w[12] + 8.0f * kY3c * x * z * w[13] +
          kY3e * (xx - yy) * w[14];
}

// Intermediates of the fp32 projection chain of one Gaussian.
struct Proj {
  float tx, ty, tz, xc, yc;
  bool clx, cly;
  float j00, j02, j11, j12;
  float s0, s1, s2;
  float qn, qw, qx, qy, qz;
  float r[9];        // Rq, row major
  float m[9];        // Rq diag(s)
  float S[6];        // Sigma: 00 01 02 11 12 22
  float T[6];        // J Rcam: row 0 then row 1
  float A, B, C, det;
  float u, v, rad;
  float ex, ey;      // half extents of the binning box
  int x0, y0, x1, y1;
};

// The fixed-order fp32 chain. Every statement below is evaluated as written:
// left-to-right sums of separately rounded products; nothing is fused except
// the two fmaf of Kahan's determinant.
__device__ bool project_chain(const abcd_camera& c, const abcd_raster_params& p, int ntx, int nty,
                              const float* mu, const float* ls, const float* q, float ologit,
                              Proj& o) {
#pragma clang fp contract(off)
  const float* R = c.R;
  o.tx = ((R[0] * mu[0] + R[1] * mu[1]) + R[2] * mu[2]) + c.t[0];
  o.ty = ((R[3] * mu[0] + R[4] * mu[1]) + R[5] * mu[2]) + c.t[1];
  o.tz = ((R[6] * mu[0] + R[7] * mu[1]) + R[8] * mu[2]) + c.t[2];
  if (!(o.tz > c.near_plane)) return false;
  const float xr = o.tx / o.tz;
  const float yr = o.ty / o.tz;
  o.u = c.fx * xr + c.cx;
  o.v = c.fy * yr + c.cy;
  const float limx = (p.guard * (0.5f * (float)c.width)) / c.fx;
  const float limy = (p.guard * (0.5f * (float)c.height)) / c.fy;
  o.clx = xr < -limx || xr > limx;
  o.cly = yr < -limy || yr > limy;
  o.xc = xr < -limx ? -limx : (xr > limx ? limx : xr);
  o.yc = yr < -limy ? -limy : (yr > limy ? limy : yr);
  o.j00 = c.fx / o.tz;
  o.j02 = -(c.fx * o.xc) / o.tz;
  o.j11 = c.fy / o.tz;
  o.j12 = -(c.fy * o.yc) / o.tz;

  o.s0 = (float)exp((double)ls[0]);
  o.s1 = (float)exp((double)ls[1]);
  o.s2 = (float)exp((double)ls[2]);

  o.qn = sqrtf(((q[0] * q[0] + q[1] * q[1]) + q[2] * q[2]) + q[3] * q[3]);
  if (!(o.qn > 0.0f) || !isfinite(o.qn)) return false;
  const float w = q[0] / o.qn, x = q[1] / o.qn, y = q[2] / o.qn, z = q[3] / o.qn;
  o.qw = w; o.qx = x; o.qy = y; o.qz = z;
  float* r = o.r;
  r[0] = 1.0f - 2.0f * (y * y + z * z);
  r[1] = 2.0f * (x * y - w * z);
  r[2] = 2.0f * (x * z + w * y);
  r[3] = 2.0f * (x * y + w * z);
  r[4] = 1.0f - 2.0f * (x * x + z * z);
  r[5] = 2.0f * (y * z - w * x);
  r[6] = 2.0f * (x * z - w * y);
  r[7] = 2.0f * (y * z + w * x);
  r[8] = 1.0f - 2.0f * (x * x + y * y);
  float* m = o.m;
  m[0] = r[0] * o.s0; m[1] = r[1] * o.s1; m[2] = r[2] * o.s2;
  m[3] = r[3] * o.s0; m[4] = r[4] * o.s1; m[5] = r[5] * o.s2;
  m[6] = r[6] * o.s0; m[7] = r[7] * o.s1; m[8] = r[8] * o.s2;
  float* S = o.S;
  S[0] = (m[0] * m[0] + m[1] * m[1]) + m[2] * m[2];
  S[1] = (m[0] * m[3] + m[1] * m[4]) + m[2] * m[5];
  S[2] = (m[0] * m[6] + m[1] * m[7]) + m[2] * m[8];
  S[3] = (m[3] * m[3] + m[4] * m[4]) + m[5] * m[5];
  S[4] = (m[3] * m[6] + m[4] * m[7]) + m[5] * m[8];
  S[5] = (m[6] * m[6] + m[7] * m[7]) + m[8] * m[8];
  float* T = o.T;
  T[0] = o.j00 * R[0] + o.j02 * R[6];
  T[1] = o.j00 * R[1] + o.j02 * R[7];
  T[2] = o.j00 * R[2] + o.j02 * R[8];
  T[3] = o.j11 * R[3] + o.j12 * R[6];
  T[4] = o.j11 * R[4] + o.j12 * R[7];
  T[5] = o.j11 * R[5] + o.j12 * R[8];
  // U = T Sigma (Sigma symmetric: S01 = S10, ...)
  const float U00 = (T[0] * S[0] + T[1] * S[1]) + T[2] * S[2];
  const float U01 = (T[0] * S[1] + T[1] * S[3]) + T[2] * S[4];
  const float U02 = (T[0] * S[2] + T[1] * S[4]) + T[2] * S[5];
  const float U10 = (T[3] * S[0] + T[4] * S[1]) + T[5] * S[2];
  const float U11 = (T[3] * S[1] + T[4] * S[3]) + T[5] * S[4];
  const float U12 = (T[3] * S[2] + T[4] * S[4]) + T[5] * S[5];
  o.A = ((U00 * T[0] + U01 * T[1]) + U02 * T[2]) + p.eps2d;
  o.B = (U00 * T[3] + U01 * T[4]) + U02 * T[5];
  o.C = ((U10 * T[3] + U11 * T[4]) + U12 * T[5]) + p.eps2d;
  // Kahan: A*C - B*B with one rounding error
  const float kw = o.B * o.B;
  const float ke = fmaf(-o.B, o.B, kw);
  const float kf = fmaf(o.A, o.C, -kw);
  o.det = kf + ke;
  if (!(o.det > 0.0f)) return false;
  const float mid = 0.5f * (o.A + o.C);
  float disc = mid * mid - o.det;
  disc = disc > 0.0f ? disc : 0.0f;
  const float lmax = mid + sqrtf(disc);
  o.rad = p.radius_sigmas * sqrtf(lmax);
  if (!isfinite(o.u) || !isfinite(o.v) || !isfinite(o.rad)) return false;
  // The binning box: the support square cut, per axis, to the extent of the
  // ellipse where alpha can reach alpha_min. A pixel offset d sees alpha =
  // o exp(-q / 2) with q = d^T Sigma^-1 d >= d_x^2 / A (and d_y^2 / C), and
  // alpha >= alpha_min needs q <= 2 ln(o / alpha_min). Bounded without
  // transcendentals, so the bound is exact fp32 arithmetic: o <= min(1,
  // e^logit), and -ln alpha_min <= (1 - e) ln 2 for alpha_min = m 2^e,
  // m in [0.5, 1). The margin is that of the blend kernels' tile test.
  int e2 = 0;
  (void)frexpf(p.alpha_min, &e2);
  const float lnb = (float)(1 - e2) * 0.6931472f;
  const float tau = 2.0f * (lnb + fminf(ologit, 0.0f));
  const float lim = tau * 1.001f + 1e-3f;
  if (!(lim > 0.0f)) return false;  // alpha_min is out of reach everywhere
  o.ex = fminf(o.rad, sqrtf(lim * o.A));
  o.ey = fminf(o.rad, sqrtf(lim * o.C));
  return tile_rect(o.u, o.v, o.ex, o.ey, ntx, nty, o.x0, o.y0, o.x1, o.y1);
}

// The geometry of one Gaussian in fp64: the 2D covariance, its inverse (the
// conic) and the intermediates its derivative needs. The binning decisions
// come from the fp32 chain above; the conic and the gradients come from here.
// For large, thin Gaussians the 2D covariance is badly conditioned (its
// determinant is far below A C, the eps2d dilation bounds only the minor
// axis), and fp32 rounding of A, B, C would be amplified by that condition
// number in the conic; fp64 arithmetic costs the HBM-bound projection
// kernels nothing measurable.
struct Geo64 {
  double tx, ty, tz, xc, yc;
  bool clx, cly;
  double j00, j02, j11, j12;
  double s[3];
  double qn, qw, qx, qy, qz;
  double r[9], m[9], S[6], T[6];
  double A, B, C, det;
};

__device__ void geom_f64(const abcd_camera& c, const abcd_raster_params& p, const float* mu,
                         const float* ls, const float* q, Geo64& o) {
  const float* R = c.R;
  const double m0 = mu[0], m1 = mu[1], m2 = mu[2];
  o.tx = (double)R[0] * m0 + (double)R[1] * m1 + (double)R[2] * m2 + (double)c.t[0];
  o.ty = (double)R[3] * m0 + (double)R[4] * m1 + (double)R[5] * m2 + (double)c.t[1];
  o.tz = (double)R[6] * m0 + (double)R[7] * m1 + (double)R[8] * m2 + (double)c.t[2];
  const double fx = c.fx, fy = c.fy;
  const double xr = o.tx / o.tz, yr = o.ty / o.tz;
  const double limx = (double)p.guard * (0.5 * (double)c.width) / fx;
  const double limy = (double)p.guard * (0.5 * (double)c.height) / fy;
  o.clx = xr < -limx || xr > limx;
  o.cly = yr < -limy || yr > limy;
  o.xc = xr < -limx ? -limx : (xr > limx ? limx : xr);
  o.yc = yr < -limy ? -limy : (yr > limy ? limy : yr);
  o.j00 = fx / o.tz;
  o.j02 = -fx * o.xc / o.tz;
  o.j11 = fy / o.tz;
  o.j12 = -fy * o.yc / o.tz;
  o.s[0] = exp((double)ls[0]);
  o.s[1] = exp((double)ls[1]);
  o.s[2] = exp((double)ls[2]);
  const double q0 = q[0], q1 = q[1], q2 = q[2], q3 = q[3];
  o.qn = sqrt(q0 * q0 + q1 * q1 + q2 * q2 + q3 * q3);
  const double w = q0 / o.qn, x = q1 / o.qn, y = q2 / o.qn, z = q3 / o.qn;
  o.qw = w; o.qx = x; o.qy = y; o.qz = z;
  double* r = o.r;
  r[0] = 1.0 - 2.0 * (y * y + z * z);
  r[1] = 2.0 * (x * y - w * z);
  r[2] = 2.0 * (x * z + w * y);
  r[3] = 2.0 * (x * y + w * z);
  r[4] = 1.0 - 2.0 * (x * x + z * z);
  r[5] = 2.0 * (y * z - w * x);
  r[6] = 2.0 * (x * z - w * y);
  r[7] = 2.0 * (y * z + w * x);
  r[8] = 1.0 - 2.0 * (x * x + y * y);
#pragma unroll
  for (int a = 0; a < 3; ++a)
#pragma unroll
    for (int b = 0; b < 3; ++b) o.m[3 * a + b] = r[3 * a + b] * o.s[b];
  const double* m = o.m;
  double* S = o.S;
  S[0] = m[0] * m[0] + m[1] * m[1] + m[2] * m[2];
  S[1] = m[0] * m[3] + m[1] * m[4] + m[2] * m[5];
  S[2] = m[0] * m[6] + m[1] * m[7] + m[2] * m[8];
  S[3] = m[3] * m[3] + m[4] * m[4] + m[5] * m[5];
  S[4] = m[3] * m[6] + m[4] * m[7] + m[5] * m[8];
  S[5] = m[6] * m[6] + m[7] * m[7] + m[8] * m[8];
  double* T = o.T;
  T[0] = o.j00 * R[0] + o.j02 * R[6];
  T[1] = o.j00 * R[1] + o.j02 * R[7];
  T[2] = o.j00 * R[2] + o.j02 * R[8];
  T[3] = o.j11 * R[3] + o.j12 * R[6];
  T[4] = o.j11 * R[4] + o.j12 * R[7];
  T[5] = o.j11 * R[5] + o.j12 * R[8];
  const double U00 = T[0] * S[0] + T[1] * S[1] + T[2] * S[2];
  const double U01 = T[0] * S[1] + T[1] * S[3] + T[2] * S[4];
  const double U02 = T[0] * S[2] + T[1] * S[4] + T[2] * S[5];
  const double U10 = T[3] * S[0] + T[4] * S[1] + T[5] * S[2];
  const double U11 = T[3] * S[1] + T[4] * S[3] + T[5] * S[4];
  const double U12 = T[3] * S[2] + T[4] * S[4] + T[5] * S[5];
  o.A = U00 * T[0] + U01 * T[1] + U02 * T[2] + (double)p.eps2d;
  o.B = U00 * T[3] + U01 * T[4] + U02 * T[5];
  o.C = U10 * T[3] + U11 * T[4] + U12 * T[5] + (double)p.eps2d;
  o.det = o.A * o.C - o.B * o.B;
}

// SH coefficients of a 64-Gaussian group are staged through LDS so that the
// global loads and stores are coalesced (each Gaussian owns 3 (D+1)^2
// consecutive floats; one thread per Gaussian would stride by 48 floats).
constexpr int kProjThreads = 64;

template <int D>
struct ShTile {
  static constexpr int kCoeffs = (D + 1) * (D + 1);
  static constexpr int kFloats = 3 * kCoeffs;
  static constexpr int kStride = kFloats + 1;  // odd stride: conflict-free LDS rows
};

// A full group issues all its loads before the first LDS write (one round
// trip to memory instead of one per element); the last, partial group loops.
template <int D>
__device__ __forceinline__ void sh_stage_in(const float* __restrict__ sh, int64_t base, int cnt,
                                            float* s) {
  using Tl = ShTile<D>;
  const float* src = sh + base * Tl::kFloats;
  if constexpr (Tl::kFloats % 4 == 0) {
    // 16-byte loads when the group's block is 16-byte aligned (a quarter of
    // the load instructions; degrees 1 and 3)
    if (cnt == kProjThreads && (reinterpret_cast<uintptr_t>(src) & 15) == 0) {
      constexpr int kVec = Tl::kFloats / 4;
      float4 v[kVec];
#pragma unroll
      for (int r = 0; r < kVec; ++r)
        v[r] = reinterpret_cast<const float4*>(src)[threadIdx.x + kProjThreads * r];
#pragma unroll
      for (int r = 0; r < kVec; ++r) {
        const int e = 4 * (threadIdx.x + kProjThreads * r);
        const int g = e / Tl::kFloats;  // the four floats share a Gaussian (kFloats % 4 == 0)
        float* row = s + g * Tl::kStride + (e - g * Tl::kFloats);
        row[0] = v[r].x;
        row[1] = v[r].y;
        row[2] = v[r].z;
        row[3] = v[r].w;
      }
      return;
    }
  }
  if (cnt == kProjThreads) {
    float v[Tl::kFloats];
#pragma unroll
    for (int r = 0; r < Tl::kFloats; ++r) v[r] = src[threadIdx.x + kProjThreads * r];
#pragma unroll
    for (int r = 0; r < Tl::kFloats; ++r) {
      const int e = threadIdx.x + kProjThreads * r;
      const int g = e / Tl::kFloats;
      s[g * Tl::kStride + (e - g * Tl::kFloats)] = v[r];
    }
    return;
  }
  for (int e = threadIdx.x; e < cnt * Tl::kFloats; e += kProjThreads) {
    const int g = e / Tl::kFloats;
    s[g * Tl::kStride + (e - g * Tl::kFloats)] = src[e];
  }
}

// Coalesced write-out (or accumulation) of a group's LDS rows to dst.
template <int D>
__device__ __forceinline__ void sh_stage_out(const float* s, int cnt, int accumulate,
                                             float* __restrict__ dst) {
  using Tl = ShTile<D>;
  if constexpr (Tl::kFloats % 4 == 0) {
    if (cnt == kProjThreads && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
      constexpr int kVec = Tl::kFloats / 4;
      float4* d4 = reinterpret_cast<float4*>(dst);
      float4 v[kVec];
#pragma unroll
      for (int r = 0; r < kVec; ++r) {
        const int e = 4 * (threadIdx.x + kProjThreads * r);
        const int g = e / Tl::kFloats;
        const float* row = s + g * Tl::kStride + (e - g * Tl::kFloats);
        v[r] = make_float4(row[0], row[1], row[2], row[3]);
      }
      if (accumulate) {
        float4 a[kVec];
#pragma unroll
        for (int r = 0; r < kVec; ++r) a[r] = d4[threadIdx.x + kProjThreads * r];
#pragma unroll
        for (int r = 0; r < kVec; ++r) {
          v[r].x += a[r].x;
          v[r].y += a[r].y;
          v[r].z += a[r].z;
          v[r].w += a[r].w;
        }
      }
#pragma unroll
      for (int r = 0; r < kVec; ++r) d4[threadIdx.x + kProjThreads * r] = v[r];
      return;
    }
  }
  if (cnt == kProjThreads) {
    float v[Tl::kFloats];
#pragma unroll
    for (int r = 0; r < Tl::kFloats; ++r) {
      const int e = threadIdx.x + kProjThreads * r;
      const int g = e / Tl::kFloats;
      v[r] = s[g * Tl::kStride + (e - g * Tl::kFloats)];
    }
    if (accumulate) {
      float a[Tl::kFloats];
#pragma unroll
      for (int r = 0; r < Tl::kFloats; ++r) a[r] = dst[threadIdx.x + kProjThreads * r];
#pragma unroll
      for (int r = 0; r < Tl::kFloats; ++r) v[r] += a[r];
    }
#pragma unroll
    for (int r = 0; r < Tl::kFloats; ++r) dst[threadIdx.x + kProjThreads * r] = v[r];
    return;
  }
  for (int e = threadIdx.x; e < cnt * Tl::kFloats; e += kProjThreads) {
    const int g = e / Tl::kFloats;
    const float v = s[g * Tl::kStride + (e - g * Tl::kFloats)];
    dst[e] = accumulate ? dst[e] + v : v;
  }
}

template <int D>
__global__ __launch_bounds__(kProjThreads) void project_kernel(
    abcd_camera cam, abcd_raster_params prm, int64_t n, int ntx, int nty, const float* __restrict__ means,
    const float* __restrict__ log_scales, const float* __restrict__ quats,
    const float* __restrict__ opacity_logits, const float* __restrict__ sh, float* __restrict__ means2d,
    float* __restrict__ conic_opacity, float* __restrict__ depth, float* __restrict__ extent,
    uint32_t* __restrict__ tiles_touched, float* __restrict__ rgb) {
  using Tl = ShTile<D>;
  __shared__ float s_sh[kProjThreads * Tl::kStride];
  const int64_t base = (int64_t)blockIdx.x * kProjThreads;
  const int cnt = (int)min<int64_t>(kProjThreads, n - base);
  const int64_t i = base + threadIdx.x;
  // every global load of the thread is issued before the first wait
  float mu[3] = {0.0f, 0.0f, 0.0f}, ls[3] = {0.0f, 0.0f, 0.0f}, ologit = 0.0f;
  float4 q4 = make_float4(1.0f, 0.0f, 0.0f, 0.0f);
  if (threadIdx.x < cnt) {
    mu[0] = means[3 * i]; mu[1] = means[3 * i + 1]; mu[2] = means[3 * i + 2];
    ls[0] = log_scales[3 * i]; ls[1] = log_scales[3 * i + 1]; ls[2] = log_scales[3 * i + 2];
    q4 = *reinterpret_cast<const float4*>(quats + 4 * i);
    ologit = opacity_logits[i];
  }
  sh_stage_in<D>(sh, base, cnt, s_sh);
  __syncthreads();
  if (threadIdx.x >= cnt) return;
  const float q[4] = {q4.x, q4.y, q4.z, q4.w};
  Proj pr;
  const bool vis = project_chain(cam, prm, ntx, nty, mu, ls, q, ologit, pr);
  if (!vis) {
    reinterpret_cast<float2*>(means2d)[i] = make_float2(0.0f, 0.0f);
    reinterpret_cast<float4*>(conic_opacity)[i] = make_float4(0, 0, 0, 0);
    depth[i] = 0.0f;
    reinterpret_cast<float2*>(extent)[i] = make_float2(0.0f, 0.0f);
    tiles_touched[i] = 0u;
    rgb[3 * i] = rgb[3 * i + 1] = rgb[3 * i + 2] = 0.0f;
    return;
  }
  Geo64 g64;
  geom_f64(cam, prm, mu, ls, q, g64);
  // the conic [[a, b], [b, c]] = inverse 2D covariance, stored as its
  // Cholesky factor [[l11, 0], [l21, l22]]: q = (l11 dx + l21 dy)^2 +
  // (l22 dy)^2 is a sum of squares, so rounding the factor to fp32 perturbs q
  // far less than rounding (a, b, c) does for a badly conditioned conic
  // (det of the conic = 1 / det, so l22 needs no subtraction)
  const double inv = 1.0 / g64.det;
  const double l11 = sqrt(g64.C * inv);
  const float ca = (float)l11, cb = (float)(-g64.B * inv / l11), cc = (float)(sqrt(inv) / l11);
  const float o = 1.0f / (1.0f + __expf(-ologit));
  float dx = mu[0] - cam.campos[0], dy = mu[1] - cam.campos[1], dz = mu[2] - cam.campos[2];
  const float dn = rsqrtf(dx * dx + dy * dy + dz * dz);
  dx *= dn; dy *= dn; dz *= dn;
  float Y[16];
  sh_eval(D, dx, dy, dz, Y, nullptr);
  const float* k = s_sh + threadIdx.x * Tl::kStride;
  float col[3] = {0.5f, 0.5f, 0.5f};
#pragma unroll
  for (int b = 0; b < Tl::kCoeffs; ++b) {
    col[0] += Y[b] * k[3 * b];
    col[1] += Y[b] * k[3 * b + 1];
    col[2] += Y[b] * k[3 * b + 2];
  }
  reinterpret_cast<float2*>(means2d)[i] = make_float2(pr.u, pr.v);
  reinterpret_cast<float4*>(conic_opacity)[i] = make_float4(ca, cb, cc, o);
  depth[i] = pr.tz;
  reinterpret_cast<float2*>(extent)[i] = make_float2(pr.ex, pr.ey);
  tiles_touched[i] = (uint32_t)((pr.x1 - pr.x0 + 1) * (pr.y1 - pr.y0 + 1));
  rgb[3 * i] = fmaxf(col[0], 0.0f);
  rgb[3 * i + 1] = fmaxf(col[1], 0.0f);
  rgb[3 * i + 2] = fmaxf(col[2], 0.0f);
}

// Chain rule from the screen-space gradients dL/d(u, v, a, b, c, o, r, g, b)
// (field q of Gaussian i at g2d[q * g2d_stride(n) + i]) to the parameters; exact derivative of the forward chain
// (guard-band clamp and colour clamp have zero derivative where active).
template <int D>
__global__ __launch_bounds__(kProjThreads) void project_bwd_kernel(
    abcd_camera cam, abcd_raster_params prm, int64_t n, int ntx, int nty,
    const float* __restrict__ means, const float* __restrict__ log_scales,
    const float* __restrict__ quats, const float* __restrict__ opacity_logits,
    const float* __restrict__ sh, const float* __restrict__ extent, const float* __restrict__ g2d,
    float* __restrict__ d_means, float* __restrict__ d_log_scales, float* __restrict__ d_quats,
    float* __restrict__ d_opacity_logits, float* __restrict__ d_sh, float* __restrict__ d_means2d,
    int accumulate) {
  using Tl = ShTile<D>;
  __shared__ float s_sh[kProjThreads * Tl::kStride];
  const int64_t base = (int64_t)blockIdx.x * kProjThreads;
  const int cnt = (int)min<int64_t>(kProjThreads, n - base);
  const int64_t i = base + threadIdx.x;
  const bool live = threadIdx.x < cnt;
  // every global load of the thread is issued before the first wait
  float mu[3] = {0, 0, 0}, ls[3] = {0, 0, 0}, ologit = 0.0f, rad = 0.0f, G[9];
  float4 q4 = make_float4(1.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
  for (int k = 0; k < 9; ++k) G[k] = 0.0f;
  if (live) {
    rad = extent[2 * i];
    mu[0] = means[3 * i]; mu[1] = means[3 * i + 1]; mu[2] = means[3 * i + 2];
    ls[0] = log_scales[3 * i]; ls[1] = log_scales[3 * i + 1]; ls[2] = log_scales[3 * i + 2];
    q4 = *reinterpret_cast<const float4*>(quats + 4 * i);
    ologit = opacity_logits[i];
#pragma unroll
    for (int k = 0; k < 9; ++k) G[k] = g2d[k * g2d_stride(n) + i];
  }
  sh_stage_in<D>(sh, base, cnt, s_sh);
  __syncthreads();
  float* kk = s_sh + threadIdx.x * Tl::kStride;  // SH in, then dL/dSH out
  float gm[3] = {0, 0, 0}, gl[3] = {0, 0, 0}, gq[4] = {0, 0, 0, 0}, gop = 0.0f;
  float gu = 0.0f, gv = 0.0f;
  Proj pr;
  bool vis = live && rad > 0.0f;
  if (vis) {
    const float q[4] = {q4.x, q4.y, q4.z, q4.w};
    vis = project_chain(cam, prm, ntx, nty, mu, ls, q, ologit, pr);
  }
  if (vis) {
    gu = G[0];
    gv = G[1];
    const float ga = G[2], gb = G[3], gc = G[4], go = G[5];
    const float gcol[3] = {G[6], G[7], G[8]};
    // the covariance part of the chain rule runs in fp64 (see geom_f64)
    Geo64 g;
    {
      const float q[4] = {q4.x, q4.y, q4.z, q4.w};
      geom_f64(cam, prm, mu, ls, q, g);
    }
    // conic Q = Sigma'^-1:  dL/dSigma' = -Q GQ Q, GQ = [[ga, gb/2], [gb/2, gc]]
    const double inv = 1.0 / g.det;
    const double qa = g.C * inv, qb = -g.B * inv, qc = g.A * inv;
    const double hb = 0.5 * gb;
    const double P00 = qa * ga + qb * hb, P01 = qa * hb + qb * gc;
    const double P10 = qb * ga + qc * hb, P11 = qb * hb + qc * gc;
    const double G00 = -(P00 * qa + P01 * qb);
    const double G01 = -0.5 * ((P00 * qb + P01 * qc) + (P10 * qa + P11 * qb));
    const double G11 = -(P10 * qb + P11 * qc);
    // Sigma' = T Sigma T^T + eps I
    const double* T = g.T;
    const double* S = g.S;
    const double Sm[9] = {S[0], S[1], S[2], S[1], S[3], S[4], S[2], S[4], S[5]};
    double GS[9];  // T^T G T
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
      for (int b = 0; b < 3; ++b)
        GS[3 * a + b] = T[a] * (G00 * T[b] + G01 * T[3 + b]) + T[3 + a] * (G01 * T[b] + G11 * T[3 + b]);
    double GT[6];  // 2 G T Sigma
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const double g0 = r == 0 ? G00 : G01, g1 = r == 0 ? G01 : G11;
#pragma unroll
      for (int b = 0; b < 3; ++b) {
        double acc = 0.0;
#pragma unroll
        for (int k = 0; k < 3; ++k) acc += (g0 * T[k] + g1 * T[3 + k]) * Sm[3 * k + b];
        GT[3 * r + b] = 2.0 * acc;
      }
    }
    // T = J Rcam
    const float* Rc = cam.R;
    const double gj00 = GT[0] * Rc[0] + GT[1] * Rc[1] + GT[2] * Rc[2];
    const double gj02 = GT[0] * Rc[6] + GT[1] * Rc[7] + GT[2] * Rc[8];
    const double gj11 = GT[3] * Rc[3] + GT[4] * Rc[4] + GT[5] * Rc[5];
    const double gj12 = GT[3] * Rc[6] + GT[4] * Rc[7] + GT[5] * Rc[8];
    // J(t), (u, v)(t)
    const double fx = cam.fx, fy = cam.fy, iz = 1.0 / g.tz, iz2 = iz * iz;
    double gtx = 0.0, gty = 0.0, gtz = 0.0;
    gtz += -fx * iz2 * gj00 - fy * iz2 * gj11 + fx * g.xc * iz2 * gj02 + fy * g.yc * iz2 * gj12;
    const double gxc = -fx * iz * gj02, gyc = -fy * iz * gj12;
    if (!g.clx) {
      gtx += gxc * iz;
      gtz -= gxc * g.tx * iz2;
    }
    if (!g.cly) {
      gty += gyc * iz;
      gtz -= gyc * g.ty * iz2;
    }
    gtx += fx * iz * gu;
    gtz -= fx * g.tx * iz2 * gu;
    gty += fy * iz * gv;
    gtz -= fy * g.ty * iz2 * gv;
#pragma unroll
    for (int k = 0; k < 3; ++k) gm[k] = (float)(Rc[k] * gtx + Rc[3 + k] * gty + Rc[6 + k] * gtz);
    // Sigma = M M^T, M = Rq diag(s)
    double GM[9];
#pragma unroll
    for (int a = 0; a < 3; ++a)
#pragma unroll
      for (int b = 0; b < 3; ++b)
        GM[3 * a + b] = 2.0 * (GS[3 * a] * g.m[b] + GS[3 * a + 1] * g.m[3 + b] +
                               GS[3 * a + 2] * g.m[6 + b]);
    double gR[9];
#pragma unroll
    for (int b = 0; b < 3; ++b) {
      double gs = 0.0;
#pragma unroll
      for (int a = 0; a < 3; ++a) {
        gs += GM[3 * a + b] * g.r[3 * a + b];
        gR[3 * a + b] = GM[3 * a + b] * g.s[b];
      }
      gl[b] = (float)(gs * g.s[b]);
    }
    // rotation entries as functions of the unit quaternion
    const double w = g.qw, x = g.qx, y = g.qy, z = g.qz;
    double gw = 0.0, gx = 0.0, gy = 0.0, gz = 0.0;
    gy += -4.0 * y * gR[0]; gz += -4.0 * z * gR[0];
    gw += -2.0 * z * gR[1]; gx += 2.0 * y * gR[1]; gy += 2.0 * x * gR[1]; gz += -2.0 * w * gR[1];
    gw += 2.0 * y * gR[2]; gx += 2.0 * z * gR[2]; gy += 2.0 * w * gR[2]; gz += 2.0 * x * gR[2];
    gw += 2.0 * z * gR[3]; gx += 2.0 * y * gR[3]; gy += 2.0 * x * gR[3]; gz += 2.0 * w * gR[3];
    gx += -4.0 * x * gR[4]; gz += -4.0 * z * gR[4];
    gw += -2.0 * x * gR[5]; gx += -2.0 * w * gR[5]; gy += 2.0 * z * gR[5]; gz += 2.0 * y * gR[5];
    gw += -2.0 * y * gR[6]; gx += 2.0 * z * gR[6]; gy += -2.0 * w * gR[6]; gz += 2.0 * x * gR[6];
    gw += 2.0 * x * gR[7]; gx += 2.0 * w * gR[7]; gy += 2.0 * z * gR[7]; gz += 2.0 * y * gR[7];
    gx += -4.0 * x * gR[8]; gy += -4.0 * y * gR[8];
    const double dotq = gw * w + gx * x + gy * y + gz * z;
    const double iq = 1.0 / g.qn;
    gq[0] = (float)((gw - w * dotq) * iq);
    gq[1] = (float)((gx - x * dotq) * iq);
    gq[2] = (float)((gy - y * dotq) * iq);
    gq[3] = (float)((gz - z * dotq) * iq);
    // opacity
    const float o = 1.0f / (1.0f + __expf(-ologit));
    gop = go * o * (1.0f - o);
    // colour: dL/dSH overwrites the thread's SH row in LDS after use
    const float d[3] = {mu[0] - cam.campos[0], mu[1] - cam.campos[1], mu[2] - cam.campos[2]};
    const float idn = 1.0f / sqrtf(d[0] * d[0] + d[1] * d[1] + d[2] * d[2]);
    const float dir[3] = {d[0] * idn, d[1] * idn, d[2] * idn};
    float Y[16];
    sh_eval(D, dir[0], dir[1], dir[2], Y, nullptr);
    float gc_[3];
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) {
      float raw = 0.5f;
#pragma unroll
      for (int b = 0; b < Tl::kCoeffs; ++b) raw += Y[b] * kk[3 * b + ch];
      gc_[ch] = raw > 0.0f ? gcol[ch] : 0.0f;
    }
    float wb[16];
#pragma unroll
    for (int b = 0; b < Tl::kCoeffs; ++b) {
      wb[b] = gc_[0] * kk[3 * b] + gc_[1] * kk[3 * b + 1] + gc_[2] * kk[3 * b + 2];
      kk[3 * b] = Y[b] * gc_[0];
      kk[3 * b + 1] = Y[b] * gc_[1];
      kk[3 * b + 2] = Y[b] * gc_[2];
    }
    float gdir[3];
    sh_grad_dot<D>(dir[0], dir[1], dir[2], wb, gdir);
    const float dd = gdir[0] * dir[0] + gdir[1] * dir[1] + gdir[2] * dir[2];
#pragma unroll
    for (int a = 0; a < 3; ++a) gm[a] += (gdir[a] - dir[a] * dd) * idn;
  } else if (live) {
#pragma unroll
    for (int k = 0; k < Tl::kFloats; ++k) kk[k] = 0.0f;
  }
  if (live) {
    float* om = d_means + 3 * i;
    float* ol = d_log_scales + 3 * i;
    float4* oq = reinterpret_cast<float4*>(d_quats) + i;
    if (accumulate) {
#pragma unroll
      for (int a = 0; a < 3; ++a) { om[a] += gm[a]; ol[a] += gl[a]; }
      const float4 q0 = *oq;
      *oq = make_float4(q0.x + gq[0], q0.y + gq[1], q0.z + gq[2], q0.w + gq[3]);
      d_opacity_logits[i] += gop;
      if (d_means2d) { d_means2d[2 * i] += gu; d_means2d[2 * i + 1] += gv; }
    } else {
#pragma unroll
      for (int a = 0; a < 3; ++a) { om[a] = gm[a]; ol[a] = gl[a]; }
      *oq = make_float4(gq[0], gq[1], gq[2], gq[3]);
      d_opacity_logits[i] = gop;
      if (d_means2d) { d_means2d[2 * i] = gu; d_means2d[2 * i + 1] = gv; }
    }
  }
  __syncthreads();
  // coalesced write-out of dL/dSH
  sh_stage_out<D>(s_sh, cnt, accumulate, d_sh + base * Tl::kFloats);
}

}  // namespace

int32_t launch_project(const abcd_camera& cam, const abcd_raster_params& prm, int64_t n,
                       const float* means, const float* log_scales, const float* quats,
                       const float* opacity_logits, const float* sh, float* means2d,
                       float* conic_opacity, float* depth, float* extent, uint32_t* tiles_touched,
                       float* rgb, hipStream_t stream) {
  if (n == 0) return ABCD_OK;
  const int64_t blocks = (n + kProjThreads - 1) / kProjThreads;
  const int ntx = tiles_x(cam.width), nty = tiles_y(cam.height);
#define ABCD_PROJ(Dg)                                                                          \
  ABCD_LAUNCH("project", project_kernel<Dg>, blocks, kProjThreads, 0, stream, cam, prm, n, ntx, \
              nty, means, log_scales, quats, opacity_logits, sh, means2d, conic_opacity, depth,  \
              extent, tiles_touched, rgb)
  switch (prm.sh_degree) {
    case 0: ABCD_PROJ(0); break;
    case 1: ABCD_PROJ(1); break;
    case 2: ABCD_PROJ(2); break;
    default: ABCD_PROJ(3); break;
  }
#undef ABCD_PROJ
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

int32_t launch_project_bwd(const abcd_camera& cam, const abcd_raster_params& prm, int64_t n,
                           const float* means, const float* log_scales, const float* quats,
                           const float* opacity_logits, const float* sh, const float* extent,
                           const float* g2d, float* d_means, float* d_log_scales, float* d_quats,
                           float* d_opacity_logits, float* d_sh, float* d_means2d,
                           int accumulate, hipStream_t stream) {
  if (n == 0) return ABCD_OK;
  const int64_t blocks = (n + kProjThreads - 1) / kProjThreads;
  const int ntx = tiles_x(cam.width), nty = tiles_y(cam.height);
#define ABCD_PROJ_BWD(Dg)                                                                    \
  ABCD_LAUNCH("project_bwd", project_bwd_kernel<Dg>, blocks, kProjThreads, 0, stream, cam, prm, \
              n, ntx, nty, means, log_scales, quats, opacity_logits, sh, extent, g2d, d_means,  \
              d_log_scales, d_quats, d_opacity_logits, d_sh, d_means2d, accumulate)
  switch (prm.sh_degree) {
    case 0: ABCD_PROJ_BWD(0); break;
    case 1: ABCD_PROJ_BWD(1); break;
    case 2: ABCD_PROJ_BWD(2); break;
    default: ABCD_PROJ_BWD(3); break;
  }
#undef ABCD_PROJ_BWD
  ABCD_HIP(hipGetLastError());
  return ABCD_OK;
}

}  // namespace abcd
