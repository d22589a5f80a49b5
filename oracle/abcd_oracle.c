/*
 * abcd_oracle.c -- CPU oracle for the ABCD active-block step.
 *
 * TEST INFRASTRUCTURE ONLY: called by the tests, the smoke check and the
 * CPU-baseline leg of the benchmark; never by the product path. Written from
 * the paper's description of the method (Method section) and from the textbook
 * definitions of the renderer it inherits from 3D Gaussian Splatting; it shares
 * no code with the GPU library.
 *
 * Build: gcc -O2 -ffp-contract=off -fopenmp -shared -fPIC (oracle/build.py).
 * -ffp-contract=off matters: the fp32 projection chain below must round every
 * operation on its own, in the order written.
 */
#include "abcd_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

static int tiles_x_of(int32_t w) { return (w + ORC_TILE - 1) / ORC_TILE; }
static int tiles_y_of(int32_t h) { return (h + ORC_TILE - 1) / ORC_TILE; }

static uint32_t f32_bits(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  return u;
}

/* ======================================================================= */
/* Projection, fp32 chain (decides culling, rectangle, depth key)            */
/* ======================================================================= */
/*
 * The operation order is the repository's numerical contract: each line is
 * one IEEE fp32 operation sequence, evaluated left to right, nothing fused.
 * The only double step is exp() of the log-scale, rounded once to fp32.
 */
static int proj_bin_one(const orc_camera* c, const orc_params* p, const float* mu,
                        const float* ls, const float* q, float ologit, float* u_out,
                        float* v_out, float* z_out, float* r_out, float ext_out[2],
                        int32_t rect[4]) {
  const float* R = c->R;
  /* view-space position */
  float tx = ((R[0] * mu[0] + R[1] * mu[1]) + R[2] * mu[2]) + c->t[0];
  float ty = ((R[3] * mu[0] + R[4] * mu[1]) + R[5] * mu[2]) + c->t[1];
  float tz = ((R[6] * mu[0] + R[7] * mu[1]) + R[8] * mu[2]) + c->t[2];
  if (!(tz > c->near_plane)) return 0;
  /* pinhole projection of the mean */
  float xr = tx / tz;
  float yr = ty / tz;
  float u = c->fx * xr + c->cx;
  float v = c->fy * yr + c->cy;
  /* Jacobian of the projection, with the ratio clamped to a guard band */
  float limx = (p->guard * (0.5f * (float)c->width)) / c->fx;
  float limy = (p->guard * (0.5f * (float)c->height)) / c->fy;
  float xc = xr < -limx ? -limx : (xr > limx ? limx : xr);
  float yc = yr < -limy ? -limy : (yr > limy ? limy : yr);
  float j00 = c->fx / tz;
  float j02 = -(c->fx * xc) / tz;
  float j11 = c->fy / tz;
  float j12 = -(c->fy * yc) / tz;
  /* scales */
  float s0 = (float)exp((double)ls[0]);
  float s1 = (float)exp((double)ls[1]);
  float s2 = (float)exp((double)ls[2]);
  /* normalised quaternion (w, x, y, z) */
  float qn = sqrtf(((q[0] * q[0] + q[1] * q[1]) + q[2] * q[2]) + q[3] * q[3]);
  if (!(qn > 0.0f) || !isfinite(qn)) return 0;
  float w = q[0] / qn, x = q[1] / qn, y = q[2] / qn, z = q[3] / qn;
  float r00 = 1.0f - 2.0f * (y * y + z * z);
  float r01 = 2.0f * (x * y - w * z);
  float r02 = 2.0f * (x * z + w * y);
  float r10 = 2.0f * (x * y + w * z);
  float r11 = 1.0f - 2.0f * (x * x + z * z);
  float r12 = 2.0f * (y * z - w * x);
  float r20 = 2.0f * (x * z - w * y);
  float r21 = 2.0f * (y * z + w * x);
  float r22 = 1.0f - 2.0f * (x * x + y * y);
  /* M = Rq diag(s) */
  float m00 = r00 * s0, m01 = r01 * s1, m02 = r02 * s2;
  float m10 = r10 * s0, m11 = r11 * s1, m12 = r12 * s2;
  float m20 = r20 * s0, m21 = r21 * s1, m22 = r22 * s2;
  /* world covariance Sigma = M M^T (upper triangle) */
  float S00 = (m00 * m00 + m01 * m01) + m02 * m02;
  float S01 = (m00 * m10 + m01 * m11) + m02 * m12;
  float S02 = (m00 * m20 + m01 * m21) + m02 * m22;
  float S11 = (m10 * m10 + m11 * m11) + m12 * m12;
  float S12 = (m10 * m20 + m11 * m21) + m12 * m22;
  float S22 = (m20 * m20 + m21 * m21) + m22 * m22;
  /* T = J Rcam (2x3) */
  float T00 = j00 * R[0] + j02 * R[6];
  float T01 = j00 * R[1] + j02 * R[7];
  float T02 = j00 * R[2] + j02 * R[8];
  float T10 = j11 * R[3] + j12 * R[6];
  float T11 = j11 * R[4] + j12 * R[7];
  float T12 = j11 * R[5] + j12 * R[8];
  /* U = T Sigma */
  float U00 = (T00 * S00 + T01 * S01) + T02 * S02;
  float U01 = (T00 * S01 + T01 * S11) + T02 * S12;
  float U02 = (T00 * S02 + T01 * S12) + T02 * S22;
  float U10 = (T10 * S00 + T11 * S01) + T12 * S02;
  float U11 = (T10 * S01 + T11 * S11) + T12 * S12;
  float U12 = (T10 * S02 + T11 * S12) + T12 * S22;
  /* 2D covariance [[A, B], [B, C]] = U T^T + eps I */
  float A = ((U00 * T00 + U01 * T01) + U02 * T02) + p->eps2d;
  float B = (U00 * T10 + U01 * T11) + U02 * T12;
  float C = ((U10 * T10 + U11 * T11) + U12 * T12) + p->eps2d;
  /* Kahan's 2x2 determinant A*C - B*B */
  float kw = B * B;
  float ke = fmaf(-B, B, kw);
  float kf = fmaf(A, C, -kw);
  float det = kf + ke;
  if (!(det > 0.0f)) return 0;
  /* largest eigenvalue and support radius */
  float mid = 0.5f * (A + C);
  float disc = mid * mid - det;
  disc = disc > 0.0f ? disc : 0.0f;
  float lmax = mid + sqrtf(disc);
  float r = p->radius_sigmas * sqrtf(lmax);
  if (!isfinite(u) || !isfinite(v) || !isfinite(r)) return 0;
  /*
   * Binning box: the support square cut per axis to the ellipse where alpha
   * can reach alpha_min. At a pixel offset d, alpha = o exp(-q/2) with
   * q = d^T Sigma^-1 d >= d_x^2 / A (and >= d_y^2 / C: a diagonal entry of
   * the inverse of a positive definite matrix is at least the reciprocal of
   * the matching entry of the matrix), so alpha >= alpha_min needs
   * d_x^2 <= A tau with tau = 2 ln(o / alpha_min). tau is bounded from above
   * with exact fp32 steps only: o = sigmoid(logit) <= min(1, e^logit), and
   * -ln(alpha_min) <= (1 - e) ln 2 where alpha_min = m 2^e, m in [0.5, 1);
   * the margin is the blend kernels' tile-test margin.
   */
  int e2 = 0;
  (void)frexpf(p->alpha_min, &e2);
  float lnb = (float)(1 - e2) * 0.6931472f;
  float tau = 2.0f * (lnb + fminf(ologit, 0.0f));
  float lim = tau * 1.001f + 1e-3f;
  if (!(lim > 0.0f)) return 0;
  float ex = fminf(r, sqrtf(lim * A));
  float ey = fminf(r, sqrtf(lim * C));
  /* tile rectangle of the box [u-ex, u+ex] x [v-ey, v+ey] */
  float tx0 = floorf((u - ex) * 0.0625f);
  float tx1 = floorf((u + ex) * 0.0625f);
  float ty0 = floorf((v - ey) * 0.0625f);
  float ty1 = floorf((v + ey) * 0.0625f);
  float ntx = (float)(tiles_x_of(c->width) - 1);
  float nty = (float)(tiles_y_of(c->height) - 1);
  if (tx0 < 0.0f) tx0 = 0.0f;
  if (ty0 < 0.0f) ty0 = 0.0f;
  if (tx1 > ntx) tx1 = ntx;
  if (ty1 > nty) ty1 = nty;
  if (tx0 > tx1 || ty0 > ty1) return 0;
  *u_out = u;
  *v_out = v;
  *z_out = tz;
  *r_out = r;
  ext_out[0] = ex;
  ext_out[1] = ey;
  rect[0] = (int32_t)tx0;
  rect[1] = (int32_t)ty0;
  rect[2] = (int32_t)tx1;
  rect[3] = (int32_t)ty1;
  return 1;
}

void orc_project_bin_f32(const orc_camera* cam, const orc_params* prm, int64_t n,
                         const float* means, const float* log_scales, const float* quats,
                         const float* opacity_logits, float* means2d, float* depth,
                         float* radius, float* extent, int32_t* rect, uint32_t* tiles_touched) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; i++) {
    float u = 0, v = 0, z = 0, r = 0, ex[2] = {0, 0};
    int32_t rc[4] = {0, 0, 0, 0};
    int vis = proj_bin_one(cam, prm, means + 3 * i, log_scales + 3 * i, quats + 4 * i,
                           opacity_logits[i], &u, &v, &z, &r, ex, rc);
    means2d[2 * i] = vis ? u : 0.0f;
    means2d[2 * i + 1] = vis ? v : 0.0f;
    depth[i] = vis ? z : 0.0f;
    radius[i] = vis ? r : 0.0f;
    extent[2 * i] = vis ? ex[0] : 0.0f;
    extent[2 * i + 1] = vis ? ex[1] : 0.0f;
    for (int k = 0; k < 4; k++) rect[4 * i + k] = vis ? rc[k] : 0;
    tiles_touched[i] = vis ? (uint32_t)((rc[2] - rc[0] + 1) * (rc[3] - rc[1] + 1)) : 0u;
  }
}

/* ======================================================================= */
/* Spherical harmonics and rotations (fp64)                                  */
/* ======================================================================= */

/*
 * Real orthonormal spherical harmonics up to degree 3, written as homogeneous
 * harmonic polynomials in the unit direction (x, y, z), index l^2 + l + m.
 * Normalisation constants are computed from their closed forms.
 */
void orc_sh_basis(const double* d, double* Y, double* G) {
  const double x = d[0], y = d[1], z = d[2];
  const double pi = 3.14159265358979323846;
  const double k0 = 0.5 * sqrt(1.0 / pi);
  const double k1 = sqrt(3.0 / (4.0 * pi));
  const double k2a = 0.5 * sqrt(15.0 / pi);
  const double k2b = 0.25 * sqrt(5.0 / pi);
  const double k2c = 0.25 * sqrt(15.0 / pi);
  const double k3a = 0.25 * sqrt(35.0 / (2.0 * pi));
  const double k3b = 0.5 * sqrt(105.0 / pi);
  const double k3c = 0.25 * sqrt(21.0 / (2.0 * pi));
  const double k3d = 0.25 * sqrt(7.0 / pi);
  const double k3e = 0.25 * sqrt(105.0 / pi);
  double y_[16], g_[48];
  memset(g_, 0, sizeof g_);
#define SETG(i, gx, gy, gz) \
  do {                      \
    g_[3 * (i)] = (gx);     \
    g_[3 * (i) + 1] = (gy); \
    g_[3 * (i) + 2] = (gz); \
  } while (0)
  /* l = 0 */
  y_[0] = k0;
  /* l = 1: y, z, x */
  y_[1] = k1 * y;
  SETG(1, 0, k1, 0);
  y_[2] = k1 * z;
  SETG(2, 0, 0, k1);
  y_[3] = k1 * x;
  SETG(3, k1, 0, 0);
  /* l = 2: xy, yz, 2z^2-x^2-y^2, xz, x^2-y^2 */
  y_[4] = k2a * x * y;
  SETG(4, k2a * y, k2a * x, 0);
  y_[5] = k2a * y * z;
  SETG(5, 0, k2a * z, k2a * y);
  y_[6] = k2b * (2 * z * z - x * x - y * y);
  SETG(6, -2 * k2b * x, -2 * k2b * y, 4 * k2b * z);
  y_[7] = k2a * x * z;
  SETG(7, k2a * z, 0, k2a * x);
  y_[8] = k2c * (x * x - y * y);
  SETG(8, 2 * k2c * x, -2 * k2c * y, 0);
  /* l = 3 */
  y_[9] = k3a * y * (3 * x * x - y * y);
  SETG(9, k3a * 6 * x * y, k3a * (3 * x * x - 3 * y * y), 0);
  y_[10] = k3b * x * y * z;
  SETG(10, k3b * y * z, k3b * x * z, k3b * x * y);
  y_[11] = k3c * y * (4 * z * z - x * x - y * y);
  SETG(11, k3c * (-2 * x * y), k3c * (4 * z * z - x * x - 3 * y * y), k3c * 8 * y * z);
  y_[12] = k3d * z * (2 * z * z - 3 * x * x - 3 * y * y);
  SETG(12, k3d * (-6 * x * z), k3d * (-6 * y * z), k3d * (6 * z * z - 3 * x * x - 3 * y * y));
  y_[13] = k3c * x * (4 * z * z - x * x - y * y);
  SETG(13, k3c * (4 * z * z - 3 * x * x - y * y), k3c * (-2 * x * y), k3c * 8 * x * z);
  y_[14] = k3e * z * (x * x - y * y);
  SETG(14, k3e * 2 * x * z, k3e * (-2 * y * z), k3e * (x * x - y * y));
  y_[15] = k3a * x * (x * x - 3 * y * y);
  SETG(15, k3a * (3 * x * x - 3 * y * y), k3a * (-6 * x * y), 0);
#undef SETG
  if (Y) memcpy(Y, y_, sizeof y_);
  if (G) memcpy(G, g_, sizeof g_);
}

void orc_quat_to_rot(const double* q, double* Rm) {
  const double w = q[0], x = q[1], y = q[2], z = q[3];
  Rm[0] = 1 - 2 * (y * y + z * z);
  Rm[1] = 2 * (x * y - w * z);
  Rm[2] = 2 * (x * z + w * y);
  Rm[3] = 2 * (x * y + w * z);
  Rm[4] = 1 - 2 * (x * x + z * z);
  Rm[5] = 2 * (y * z - w * x);
  Rm[6] = 2 * (x * z - w * y);
  Rm[7] = 2 * (y * z + w * x);
  Rm[8] = 1 - 2 * (x * x + y * y);
}

/* derivative of each rotation entry with respect to (w, x, y, z) */
static void quat_rot_jacobian(const double* q, double dR[9][4]) {
  const double w = q[0], x = q[1], y = q[2], z = q[3];
  const double t[9][4] = {
      {0, 0, -4 * y, -4 * z},         /* 1 - 2(y^2 + z^2) */
      {-2 * z, 2 * y, 2 * x, -2 * w}, /* 2(xy - wz) */
      {2 * y, 2 * z, 2 * w, 2 * x},   /* 2(xz + wy) */
      {2 * z, 2 * y, 2 * x, 2 * w},   /* 2(xy + wz) */
      {0, -4 * x, 0, -4 * z},         /* 1 - 2(x^2 + z^2) */
      {-2 * x, -2 * w, 2 * z, 2 * y}, /* 2(yz - wx) */
      {-2 * y, 2 * z, -2 * w, 2 * x}, /* 2(xz - wy) */
      {2 * x, 2 * w, 2 * z, 2 * y},   /* 2(yz + wx) */
      {0, -4 * x, -4 * y, 0},         /* 1 - 2(x^2 + y^2) */
  };
  memcpy(dR, t, sizeof t);
}

/* ======================================================================= */
/* Projection, fp64 values and their intermediates                           */
/* ======================================================================= */

typedef struct {
  double t[3];
  double xr, yr, u, v, xc, yc;
  int clamp_x, clamp_y;
  double J[2][3];
  double s[3];
  double qnorm, qh[4];
  double Rq[9], M[9], S[9]; /* row major 3x3 */
  double T[2][3];
  double A, B, C, det;
  double a, b, c; /* conic */
  double o;
  double d[3], dnorm, dir[3];
  double Y[16], Yg[48];
  double raw[3], rgb[3];
} gauss64;

static void proj_values_one(const orc_camera* cm, const orc_params* p, const float* mu,
                            const float* ls, const float* q, float logit, const float* sh,
                            gauss64* g) {
  double Rc[9];
  for (int i = 0; i < 9; i++) Rc[i] = cm->R[i];
  for (int i = 0; i < 3; i++)
    g->t[i] = Rc[3 * i] * mu[0] + Rc[3 * i + 1] * mu[1] + Rc[3 * i + 2] * mu[2] + cm->t[i];
  const double fx = cm->fx, fy = cm->fy, tz = g->t[2];
  g->xr = g->t[0] / tz;
  g->yr = g->t[1] / tz;
  g->u = fx * g->xr + cm->cx;
  g->v = fy * g->yr + cm->cy;
  const double limx = (double)p->guard * 0.5 * cm->width / fx;
  const double limy = (double)p->guard * 0.5 * cm->height / fy;
  g->clamp_x = g->xr < -limx || g->xr > limx;
  g->clamp_y = g->yr < -limy || g->yr > limy;
  g->xc = g->xr < -limx ? -limx : (g->xr > limx ? limx : g->xr);
  g->yc = g->yr < -limy ? -limy : (g->yr > limy ? limy : g->yr);
  memset(g->J, 0, sizeof g->J);
  g->J[0][0] = fx / tz;
  g->J[0][2] = -fx * g->xc / tz;
  g->J[1][1] = fy / tz;
  g->J[1][2] = -fy * g->yc / tz;

  for (int i = 0; i < 3; i++) g->s[i] = exp((double)ls[i]);
  g->qnorm = sqrt((double)q[0] * q[0] + (double)q[1] * q[1] + (double)q[2] * q[2] +
                  (double)q[3] * q[3]);
  for (int i = 0; i < 4; i++) g->qh[i] = q[i] / g->qnorm;
  orc_quat_to_rot(g->qh, g->Rq);
  for (int i = 0; i < 3; i++)
    for (int j = 0; j < 3; j++) g->M[3 * i + j] = g->Rq[3 * i + j] * g->s[j];
  for (int i = 0; i < 3; i++)
    for (int j = 0; j < 3; j++) {
      double acc = 0;
      for (int k = 0; k < 3; k++) acc += g->M[3 * i + k] * g->M[3 * j + k];
      g->S[3 * i + j] = acc;
    }
  for (int i = 0; i < 2; i++)
    for (int j = 0; j < 3; j++) {
      double acc = 0;
      for (int k = 0; k < 3; k++) acc += g->J[i][k] * Rc[3 * k + j];
      g->T[i][j] = acc;
    }
  double Sp[2][2];
  for (int i = 0; i < 2; i++)
    for (int j = 0; j < 2; j++) {
      double acc = 0;
      for (int k = 0; k < 3; k++)
        for (int l = 0; l < 3; l++) acc += g->T[i][k] * g->S[3 * k + l] * g->T[j][l];
      Sp[i][j] = acc;
    }
  g->A = Sp[0][0] + p->eps2d;
  g->B = Sp[0][1];
  g->C = Sp[1][1] + p->eps2d;
  g->det = g->A * g->C - g->B * g->B;
  g->a = g->C / g->det;
  g->b = -g->B / g->det;
  g->c = g->A / g->det;
  g->o = 1.0 / (1.0 + exp(-(double)logit));

  for (int i = 0; i < 3; i++) g->d[i] = (double)mu[i] - (double)cm->campos[i];
  g->dnorm = sqrt(g->d[0] * g->d[0] + g->d[1] * g->d[1] + g->d[2] * g->d[2]);
  for (int i = 0; i < 3; i++) g->dir[i] = g->d[i] / g->dnorm;
  orc_sh_basis(g->dir, g->Y, g->Yg);
  const int nc = (p->sh_degree + 1) * (p->sh_degree + 1);
  for (int ch = 0; ch < 3; ch++) {
    double acc = 0;
    for (int i = 0; i < nc; i++) acc += g->Y[i] * sh[3 * i + ch];
    g->raw[ch] = acc + 0.5;
    g->rgb[ch] = g->raw[ch] > 0 ? g->raw[ch] : 0.0;
  }
}

void orc_project_values_f64(const orc_camera* cam, const orc_params* prm, int64_t n,
                            const float* means, const float* log_scales, const float* quats,
                            const float* opacity_logits, const float* sh,
                            const uint32_t* tiles_touched, double* means2d, double* conic,
                            double* opacity, double* rgb) {
  const int nc = (prm->sh_degree + 1) * (prm->sh_degree + 1);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; i++) {
    if (tiles_touched[i] == 0) {
      means2d[2 * i] = means2d[2 * i + 1] = 0;
      conic[3 * i] = conic[3 * i + 1] = conic[3 * i + 2] = 0;
      opacity[i] = 0;
      rgb[3 * i] = rgb[3 * i + 1] = rgb[3 * i + 2] = 0;
      continue;
    }
    gauss64 g;
    proj_values_one(cam, prm, means + 3 * i, log_scales + 3 * i, quats + 4 * i,
                    opacity_logits[i], sh + (int64_t)3 * nc * i, &g);
    means2d[2 * i] = g.u;
    means2d[2 * i + 1] = g.v;
    conic[3 * i] = g.a;
    conic[3 * i + 1] = g.b;
    conic[3 * i + 2] = g.c;
    opacity[i] = g.o;
    for (int ch = 0; ch < 3; ch++) rgb[3 * i + ch] = g.rgb[ch];
  }
}

/* ======================================================================= */
/* Binning                                                                   */
/* ======================================================================= */

int64_t orc_count_isect(int64_t n, const uint32_t* tiles_touched) {
  int64_t m = 0;
  for (int64_t i = 0; i < n; i++) m += tiles_touched[i];
  return m;
}

typedef struct {
  uint64_t key;
  uint32_t idx;
} isect;

static int isect_cmp(const void* pa, const void* pb) {
  const isect* a = (const isect*)pa;
  const isect* b = (const isect*)pb;
  if (a->key != b->key) return a->key < b->key ? -1 : 1;
  if (a->idx != b->idx) return a->idx < b->idx ? -1 : 1;
  return 0;
}

void orc_bin(int32_t width, int32_t height, int64_t n, const float* depth, const int32_t* rect,
             const uint32_t* tiles_touched, uint64_t* keys, uint32_t* values,
             uint32_t* tile_ranges) {
  /* Every (tile, Gaussian) pair of the support rectangles, ordered by
   * (key, index) with key = tile << 32 | depth bits. The tile is the key's
   * high part, so that order is: tiles in increasing order, and within a tile
   * its Gaussians by (depth bits, index). The pairs are first grouped by tile
   * (a counting pass over the rectangles, then placement in index order) and
   * each tile's group is sorted on its own, which gives the same sequence as
   * one sort of all pairs and lets the tiles sort in parallel. */
  const int ntx = tiles_x_of(width), nty = tiles_y_of(height);
  const int64_t ntiles = (int64_t)ntx * nty;
  const int64_t m = orc_count_isect(n, tiles_touched);
  int64_t* start = (int64_t*)calloc((size_t)ntiles + 1, sizeof(int64_t));
  int64_t* fill = (int64_t*)malloc(sizeof(int64_t) * (size_t)(ntiles + 1));
  for (int64_t i = 0; i < n; i++) {
    if (tiles_touched[i] == 0) continue;
    const int32_t* rc = rect + 4 * i;
    for (int ty = rc[1]; ty <= rc[3]; ty++)
      for (int tx = rc[0]; tx <= rc[2]; tx++) start[(int64_t)ty * ntx + tx + 1]++;
  }
  for (int64_t t = 0; t < ntiles; t++) start[t + 1] += start[t];
  memcpy(fill, start, sizeof(int64_t) * (size_t)(ntiles + 1));
  isect* list = (isect*)malloc(sizeof(isect) * (size_t)(m > 0 ? m : 1));
  for (int64_t i = 0; i < n; i++) {
    if (tiles_touched[i] == 0) continue;
    const int32_t* rc = rect + 4 * i;
    for (int ty = rc[1]; ty <= rc[3]; ty++)
      for (int tx = rc[0]; tx <= rc[2]; tx++) {
        const uint64_t tile = (uint64_t)ty * ntx + tx;
        const int64_t k = fill[tile]++;
        list[k].key = (tile << 32) | f32_bits(depth[i]);
        list[k].idx = (uint32_t)i;
      }
  }
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t t = 0; t < ntiles; t++)
    qsort(list + start[t], (size_t)(start[t + 1] - start[t]), sizeof(isect), isect_cmp);
  for (int64_t t = 0; t < ntiles; t++) {
    tile_ranges[2 * t] = (uint32_t)start[t];
    tile_ranges[2 * t + 1] = (uint32_t)start[t + 1];
  }
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < m; j++) {
    keys[j] = list[j].key;
    values[j] = list[j].idx;
  }
  free(list);
  free(fill);
  free(start);
}

/* ======================================================================= */
/* Forward rasterisation and composite (fp64)                                */
/* ======================================================================= */

static int near_rel(double x, double ref, double rel) {
  return rel > 0 && fabs(x - ref) <= rel * fabs(ref);
}

void orc_render_fwd(const orc_camera* cam, const orc_params* prm, const uint32_t* tile_ranges,
                    const uint32_t* values, const double* means2d, const double* conic,
                    const double* opacity, const double* rgb, const double* F, const double* B,
                    double* out, double* final_T, uint32_t* last, uint64_t* n_blends,
                    double rel_margin, double f32_kappa, uint8_t* knife, double* t_stop) {
  const int W = cam->width, H = cam->height;
  const int ntx = tiles_x_of(W);
  const int64_t npix = (int64_t)W * H;
  uint64_t total = 0;
#pragma omp parallel for schedule(dynamic, 64) reduction(+ : total)
  for (int64_t pix = 0; pix < npix; pix++) {
    const int px = (int)(pix % W), py = (int)(pix / W);
    const int64_t tile = (int64_t)(py / ORC_TILE) * ntx + px / ORC_TILE;
    const uint32_t start = tile_ranges[2 * tile], end = tile_ranges[2 * tile + 1];
    const double cxp = px + 0.5, cyp = py + 0.5;
    double T = 1.0, Cr = 0, Cg = 0, Cb = 0, tst = 0;
    uint32_t lst = 0;
    int kn = 0;
    double f[4] = {0, 0, 0, 0}, bb[4] = {0, 0, 0, 0};
    if (F) memcpy(f, F + 4 * pix, sizeof f);
    if (B) memcpy(bb, B + 4 * pix, sizeof bb);
    /* weight of the active render in the composited image: 1 - F_alpha */
    const double vis = prm->fb_stop ? 1.0 - f[3] : 1.0;
    /* relative error bound of the transmittance a fp32 walk would hold (with
     * f32_kappa > 0): one rounding per blend plus the alpha errors below */
    double errT = 0.0;
    for (uint32_t k = start; k < end; k++) {
      const uint32_t g = values[k];
      const double dx = cxp - means2d[2 * g], dy = cyp - means2d[2 * g + 1];
      const double a = conic[3 * g], b = conic[3 * g + 1], c = conic[3 * g + 2];
      const double power = -0.5 * (a * dx * dx + c * dy * dy) - b * dx * dy;
      const double terms = 0.5 * (fabs(a) * dx * dx + fabs(c) * dy * dy) + fabs(b * dx * dy);
      if (rel_margin > 0 && terms > 0 && fabs(power) <= rel_margin * terms) kn = 1;
      if (power > 0) continue;
      /* margin of the alpha decisions: rel_margin, plus (f32_kappa > 0) a
       * bound on the relative error of alpha evaluated in fp32 from a
       * fp32-rounded Cholesky factor L of the conic, q = (l11 dx + l21 dy)^2 +
       * (l22 dy)^2: each product and the factor carry a relative rounding of
       * 2^-24, so q moves by at most a small multiple of 2^-24 times
       * |e1| (|l11 dx| + |l21 dy|) + |e2| |l22 dy| + q, and alpha = o e^(-q/2)
       * by half of that, relatively. Large where the two products of e1
       * nearly cancel (long thin splats seen along their major axis). */
      double da = rel_margin;
      if (f32_kappa > 0) {
        const double l11 = sqrt(a), l21 = b / l11;
        const double l22 = sqrt(fmax(c - l21 * l21, 0.0));
        const double e1 = l11 * dx + l21 * dy, e2 = l22 * dy;
        da += f32_kappa * 0x1p-24 *
              (fabs(e1) * (fabs(l11 * dx) + fabs(l21 * dy)) + fabs(e2) * fabs(l22 * dy) +
               e1 * e1 + e2 * e2);
      }
      const double araw = opacity[g] * exp(power);
      if (near_rel(araw, prm->alpha_max, da)) kn = 1;
      const double alpha = araw < prm->alpha_max ? araw : prm->alpha_max;
      if (near_rel(alpha, prm->alpha_min, da)) kn = 1;
      if (alpha < prm->alpha_min) continue;
      const double Tn = T * (1.0 - alpha);
      /* the stop decision: rel_margin alone, or with f32_kappa > 0 the error
       * bound of the fp32 transmittance including this entry's alpha */
      const double dstep = alpha / (1.0 - alpha) * da;
      const double dT = f32_kappa > 0 ? rel_margin + errT + dstep + 4 * 0x1p-24 : rel_margin;
      if (near_rel(vis * Tn, prm->t_min, dT)) kn = 1;
      if (vis * Tn < prm->t_min) {
        tst = T;
        break;
      }
      errT += dstep + 2 * 0x1p-24;
      Cr += rgb[3 * g] * alpha * T;
      Cg += rgb[3 * g + 1] * alpha * T;
      Cb += rgb[3 * g + 2] * alpha * T;
      T = Tn;
      lst = k - start + 1;
      total++;
    }
    /* premultiplied composite out = F over A over B, A = (C, 1 - T) */
    const double sfr = 1.0 - f[3];
    out[4 * pix + 0] = f[0] + sfr * (Cr + T * bb[0]);
    out[4 * pix + 1] = f[1] + sfr * (Cg + T * bb[1]);
    out[4 * pix + 2] = f[2] + sfr * (Cb + T * bb[2]);
    out[4 * pix + 3] = f[3] + sfr * (1.0 - T * (1.0 - bb[3]));
    final_T[pix] = T;
    last[pix] = lst;
    if (knife) knife[pix] = (uint8_t)kn;
    if (t_stop) t_stop[pix] = tst;
  }
  if (n_blends) *n_blends = total;
}

/* ======================================================================= */
/* Backward, per pixel (fp64)                                               */
/* ======================================================================= */

typedef struct {
  uint32_t g;
  double alpha, T, e, dx, dy;
  int clamped;
} blended;

void orc_render_bwd_2d(const orc_camera* cam, const orc_params* prm, int64_t n,
                       const uint32_t* tile_ranges, const uint32_t* values,
                       const double* means2d, const double* conic, const double* opacity,
                       const double* rgb, const double* F, const double* B,
                       const double* dL_dout, double* g2d) {
  const int W = cam->width, H = cam->height;
  const int ntx = tiles_x_of(W);
  const int64_t npix = (int64_t)W * H;
  memset(g2d, 0, sizeof(double) * 9 * (size_t)n);
#pragma omp parallel
  {
    size_t cap = 256;
    blended* bl = (blended*)malloc(sizeof(blended) * cap);
#pragma omp for schedule(dynamic, 64)
    for (int64_t pix = 0; pix < npix; pix++) {
      const int px = (int)(pix % W), py = (int)(pix / W);
      const int64_t tile = (int64_t)(py / ORC_TILE) * ntx + px / ORC_TILE;
      const uint32_t start = tile_ranges[2 * tile], end = tile_ranges[2 * tile + 1];
      const double cxp = px + 0.5, cyp = py + 0.5;
      double f[4] = {0, 0, 0, 0}, bb[4] = {0, 0, 0, 0};
      if (F) memcpy(f, F + 4 * pix, sizeof f);
      if (B) memcpy(bb, B + 4 * pix, sizeof bb);
      const double vis = prm->fb_stop ? 1.0 - f[3] : 1.0;
      /* replay the forward walk, recording every blended entry */
      size_t nb = 0;
      double T = 1.0;
      for (uint32_t k = start; k < end; k++) {
        const uint32_t g = values[k];
        const double dx = cxp - means2d[2 * g], dy = cyp - means2d[2 * g + 1];
        const double a = conic[3 * g], b = conic[3 * g + 1], c = conic[3 * g + 2];
        const double power = -0.5 * (a * dx * dx + c * dy * dy) - b * dx * dy;
        if (power > 0) continue;
        const double e = exp(power);
        const double araw = opacity[g] * e;
        const int clamped = araw > prm->alpha_max;
        const double alpha = clamped ? prm->alpha_max : araw;
        if (alpha < prm->alpha_min) continue;
        const double Tn = T * (1.0 - alpha);
        if (vis * Tn < prm->t_min) break;
        if (nb == cap) {
          cap *= 2;
          bl = (blended*)realloc(bl, sizeof(blended) * cap);
        }
        bl[nb].g = g;
        bl[nb].alpha = alpha;
        bl[nb].T = T;
        bl[nb].e = e;
        bl[nb].dx = dx;
        bl[nb].dy = dy;
        bl[nb].clamped = clamped;
        nb++;
        T = Tn;
      }
      /* gradients of out = F over (C, 1-T) over B with respect to C and T */
      const double* G = dL_dout + 4 * pix;
      const double sfr = 1.0 - f[3];
      const double gC[3] = {sfr * G[0], sfr * G[1], sfr * G[2]};
      const double gT = sfr * (G[0] * bb[0] + G[1] * bb[1] + G[2] * bb[2] - G[3] * (1.0 - bb[3]));
      /* walk back: R = colour behind entry k, S = product of (1-alpha) behind k */
      double Rr[3] = {0, 0, 0}, S = 1.0;
      for (size_t j = nb; j-- > 0;) {
        const blended* e = &bl[j];
        const uint32_t g = e->g;
        const double* col = rgb + 3 * g;
        double grad[9] = {0, 0, 0, 0, 0, 0, 0, 0, 0};
        for (int ch = 0; ch < 3; ch++) grad[6 + ch] = e->alpha * e->T * gC[ch];
        double dL_dalpha = 0;
        for (int ch = 0; ch < 3; ch++) dL_dalpha += e->T * (col[ch] - Rr[ch]) * gC[ch];
        dL_dalpha -= e->T * S * gT; /* d T_final / d alpha = -T_final / (1 - alpha) */
        if (!e->clamped) {
          const double a = conic[3 * g], b = conic[3 * g + 1], c = conic[3 * g + 2];
          const double dL_dpow = e->alpha * dL_dalpha;
          grad[5] = e->e * dL_dalpha;
          grad[0] = dL_dpow * (a * e->dx + b * e->dy);
          grad[1] = dL_dpow * (b * e->dx + c * e->dy);
          grad[2] = dL_dpow * (-0.5 * e->dx * e->dx);
          grad[3] = dL_dpow * (-e->dx * e->dy);
          grad[4] = dL_dpow * (-0.5 * e->dy * e->dy);
        }
        for (int q = 0; q < 9; q++) {
#pragma omp atomic
          g2d[9 * (int64_t)g + q] += grad[q];
        }
        for (int ch = 0; ch < 3; ch++) Rr[ch] = col[ch] * e->alpha + (1.0 - e->alpha) * Rr[ch];
        S *= 1.0 - e->alpha;
      }
    }
    free(bl);
  }
}

/* ======================================================================= */
/* Backward, per Gaussian chain rule (fp64)                                  */
/* ======================================================================= */

void orc_project_bwd(const orc_camera* cm, const orc_params* p, int64_t n, const float* means,
                     const float* log_scales, const float* quats, const float* opacity_logits,
                     const float* sh, const uint32_t* tiles_touched, const double* g2d,
                     double* d_means, double* d_log_scales, double* d_quats,
                     double* d_opacity_logits, double* d_sh) {
  const int nc = (p->sh_degree + 1) * (p->sh_degree + 1);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; i++) {
    double* gmu = d_means + 3 * i;
    double* gls = d_log_scales + 3 * i;
    double* gq = d_quats + 4 * i;
    double* gsh = d_sh + (int64_t)3 * nc * i;
    for (int k = 0; k < 3; k++) gmu[k] = gls[k] = 0;
    for (int k = 0; k < 4; k++) gq[k] = 0;
    for (int k = 0; k < 3 * nc; k++) gsh[k] = 0;
    d_opacity_logits[i] = 0;
    if (tiles_touched[i] == 0) continue;

    const float* shi = sh + (int64_t)3 * nc * i;
    gauss64 g;
    proj_values_one(cm, p, means + 3 * i, log_scales + 3 * i, quats + 4 * i, opacity_logits[i],
                    shi, &g);
    const double* G = g2d + 9 * i;
    const double gu = G[0], gv = G[1], ga = G[2], gb = G[3], gc = G[4], go = G[5];
    double Rc[9];
    for (int k = 0; k < 9; k++) Rc[k] = cm->R[k];

    /* conic Q = inverse of Sigma': dL/dSigma' = -Q GQ Q, GQ symmetric */
    const double Q[2][2] = {{g.a, g.b}, {g.b, g.c}};
    const double GQ[2][2] = {{ga, 0.5 * gb}, {0.5 * gb, gc}};
    double QG[2][2], GS2[2][2];
    for (int r = 0; r < 2; r++)
      for (int c = 0; c < 2; c++) QG[r][c] = Q[r][0] * GQ[0][c] + Q[r][1] * GQ[1][c];
    for (int r = 0; r < 2; r++)
      for (int c = 0; c < 2; c++) GS2[r][c] = -(QG[r][0] * Q[0][c] + QG[r][1] * Q[1][c]);

    /* Sigma' = T Sigma T^T + eps I */
    double GS3[3][3], GT[2][3];
    for (int r = 0; r < 3; r++)
      for (int c = 0; c < 3; c++) {
        double acc = 0;
        for (int k = 0; k < 2; k++)
          for (int l = 0; l < 2; l++) acc += g.T[k][r] * GS2[k][l] * g.T[l][c];
        GS3[r][c] = acc;
      }
    for (int r = 0; r < 2; r++)
      for (int c = 0; c < 3; c++) {
        double acc = 0;
        for (int k = 0; k < 2; k++)
          for (int l = 0; l < 3; l++) acc += GS2[r][k] * g.T[k][l] * g.S[3 * l + c];
        GT[r][c] = 2.0 * acc;
      }
    /* T = J Rcam */
    double GJ[2][3];
    for (int r = 0; r < 2; r++)
      for (int c = 0; c < 3; c++) {
        double acc = 0;
        for (int k = 0; k < 3; k++) acc += GT[r][k] * Rc[3 * c + k];
        GJ[r][c] = acc;
      }
    /* J(t) and (u, v)(t) */
    const double fx = cm->fx, fy = cm->fy;
    const double tx = g.t[0], ty = g.t[1], tz = g.t[2];
    double gt[3] = {0, 0, 0};
    gt[2] += -fx / (tz * tz) * GJ[0][0] - fy / (tz * tz) * GJ[1][1];
    gt[2] += fx * g.xc / (tz * tz) * GJ[0][2] + fy * g.yc / (tz * tz) * GJ[1][2];
    const double gxc = -fx / tz * GJ[0][2];
    const double gyc = -fy / tz * GJ[1][2];
    if (!g.clamp_x) {
      gt[0] += gxc / tz;
      gt[2] += -gxc * tx / (tz * tz);
    }
    if (!g.clamp_y) {
      gt[1] += gyc / tz;
      gt[2] += -gyc * ty / (tz * tz);
    }
    gt[0] += fx / tz * gu;
    gt[2] += -fx * tx / (tz * tz) * gu;
    gt[1] += fy / tz * gv;
    gt[2] += -fy * ty / (tz * tz) * gv;
    /* t = Rcam mu + tcam */
    for (int k = 0; k < 3; k++) gmu[k] += Rc[k] * gt[0] + Rc[3 + k] * gt[1] + Rc[6 + k] * gt[2];

    /* Sigma = M M^T, M = Rq diag(s) */
    double GM[3][3];
    for (int r = 0; r < 3; r++)
      for (int c = 0; c < 3; c++) {
        double acc = 0;
        for (int k = 0; k < 3; k++) acc += GS3[r][k] * g.M[3 * k + c];
        GM[r][c] = 2.0 * acc;
      }
    double gRq[9];
    for (int c = 0; c < 3; c++) {
      double gs = 0;
      for (int r = 0; r < 3; r++) {
        gs += GM[r][c] * g.Rq[3 * r + c];
        gRq[3 * r + c] = GM[r][c] * g.s[c];
      }
      gls[c] = gs * g.s[c];
    }
    /* rotation of the normalised quaternion, then the normalisation */
    double dR[9][4];
    quat_rot_jacobian(g.qh, dR);
    double gqh[4] = {0, 0, 0, 0};
    for (int e = 0; e < 9; e++)
      for (int k = 0; k < 4; k++) gqh[k] += gRq[e] * dR[e][k];
    const double dotq = gqh[0] * g.qh[0] + gqh[1] * g.qh[1] + gqh[2] * g.qh[2] + gqh[3] * g.qh[3];
    for (int k = 0; k < 4; k++) gq[k] = (gqh[k] - g.qh[k] * dotq) / g.qnorm;

    /* opacity = sigmoid(logit) */
    d_opacity_logits[i] = go * g.o * (1.0 - g.o);

    /* colour = max(0, sum_i Y_i(dir) k_i + 0.5) */
    double gdir[3] = {0, 0, 0};
    for (int ch = 0; ch < 3; ch++) {
      if (!(g.raw[ch] > 0)) continue;
      const double gcol = G[6 + ch];
      for (int b = 0; b < nc; b++) {
        gsh[3 * b + ch] = g.Y[b] * gcol;
        for (int k = 0; k < 3; k++) gdir[k] += gcol * shi[3 * b + ch] * g.Yg[3 * b + k];
      }
    }
    const double dd = gdir[0] * g.dir[0] + gdir[1] * g.dir[1] + gdir[2] * g.dir[2];
    for (int k = 0; k < 3; k++) gmu[k] += (gdir[k] - g.dir[k] * dd) / g.dnorm;
  }
}

/* ======================================================================= */
/* "Over" collapse of cached renders (fp64)                                  */
/* ======================================================================= */

double orc_half_to_double(uint16_t h) {
  const int sign = h >> 15, ex = (h >> 10) & 31, man = h & 1023;
  double v;
  if (ex == 0)
    v = ldexp((double)man, -24); /* subnormal: man * 2^-24 */
  else if (ex == 31)
    v = man ? NAN : INFINITY;
  else
    v = ldexp((double)(1024 + man), ex - 25); /* (1 + man/1024) * 2^(ex-15) */
  return sign ? -v : v;
}

void orc_composite(int32_t width, int32_t height, int32_t k, const uint16_t* images,
                   const int32_t* order, int32_t n_front, double* F, double* B,
                   int32_t accumulate, double stop_t, double rel_margin, uint8_t* knife) {
  const int64_t npix = (int64_t)width * height;
#pragma omp parallel for schedule(static)
  for (int64_t pix = 0; pix < npix; pix++) {
    /* acc[0] = F, acc[1] = B; a left fold of premultiplied "over" */
    double acc[2][4] = {{0, 0, 0, 0}, {0, 0, 0, 0}};
    if (accumulate) {
      memcpy(acc[0], F + 4 * pix, sizeof acc[0]);
      memcpy(acc[1], B + 4 * pix, sizeof acc[1]);
    }
    int kn = 0;
    for (int j = 0; j < k; j++) {
      const int l = j < n_front ? 0 : 1;
      if (stop_t > 0) {
        /* the largest weight this layer could still get in the final image */
        const double vis = (1.0 - acc[l][3]) * (l == 1 ? 1.0 - acc[0][3] : 1.0);
        if (near_rel(vis, stop_t, rel_margin)) kn = 1;
        if (vis < stop_t) continue;
      }
      const uint16_t* px = images + ((int64_t)order[j] * npix + pix) * 4;
      double x[4];
      for (int c = 0; c < 4; c++) x[c] = orc_half_to_double(px[c]);
      /* acc = acc over x (premultiplied): acc + (1 - acc_alpha) x */
      const double s = 1.0 - acc[l][3];
      for (int c = 0; c < 4; c++) acc[l][c] = acc[l][c] + s * x[c];
    }
    memcpy(F + 4 * pix, acc[0], sizeof acc[0]);
    memcpy(B + 4 * pix, acc[1], sizeof acc[1]);
    if (knife) knife[pix] = (uint8_t)kn;
  }
}

void orc_adam(int64_t n, double* theta, const double* g, double* m, double* v, double lr,
              double b1, double b2, double eps, int64_t t) {
  const double c1 = 1.0 - pow(b1, (double)t), c2 = 1.0 - pow(b2, (double)t);
  for (int64_t i = 0; i < n; i++) {
    m[i] = b1 * m[i] + (1.0 - b1) * g[i];
    v[i] = b2 * v[i] + (1.0 - b2) * g[i] * g[i];
    const double mhat = m[i] / c1, vhat = v[i] / c2;
    theta[i] = theta[i] - lr * mhat / (sqrt(vhat) + eps);
  }
}
