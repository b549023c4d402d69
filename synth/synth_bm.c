/* synth_bm.c - Box-Muller transform over arrays of uniforms (Box & Muller,
 * 1958): z0 = sqrt(-2 ln a) cos(2 pi b), z1 = sqrt(-2 ln a) sin(2 pi b).
 * Compiled on its own with vector math so that the loops run on the C
 * library's SIMD log/cos/sin (the rest of the generator is built without
 * fast-math).  The generator library is built once and used by every
 * consumer, so all of them see the same values.  The cosine and sine loops
 * are separate: a joint sincos has no SIMD variant. */
#include <math.h>

void synth_box_muller(const double *restrict a, const double *restrict b, double *restrict r,
                      double *restrict t, double *restrict z, int n) {
  for (int i = 0; i < n; ++i) {
    r[i] = sqrt(-2.0 * log(a[i]));
    t[i] = 6.283185307179586476925286766559 * b[i];
  }
  for (int i = 0; i < n; ++i) z[2 * i] = r[i] * cos(t[i]);
  for (int i = 0; i < n; ++i) z[2 * i + 1] = r[i] * sin(t[i]);
}
