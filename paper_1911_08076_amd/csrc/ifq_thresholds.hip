// Expansion of compact per-channel thresholds (Eq. 8, uniform quantizer) into
// the records the conv epilogues read, {s, T_1 .. T_nq} per channel, on the
// device: one thread per channel, fp64 in the order the header states (the
// product i * base' rounded on its own, then the sum, then the floor of the
// signed value), so a layer can keep two doubles per channel resident and
// expand them where it runs.
#include <hip/hip_runtime.h>

#include "ifq_internal.h"

namespace ifq {
namespace {

__global__ __launch_bounds__(256) void expand_thresholds(const ifq_thr_compact* recs, int c_out,
                                                         int nq, double bound, int32_t* thr) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= c_out) return;
  const ifq_thr_compact r = recs[c];
  int32_t* o = thr + (int64_t)c * (nq + 1);
  if (r.s == 0) {
    // gamma == 0: the constant code cstar, as the table fold encodes it
    o[0] = 1;
    for (int i = 1; i <= nq; ++i) o[i] = i <= r.cstar ? (int32_t)(-bound - 1.0) : (int32_t)bound;
    return;
  }
  o[0] = r.s > 0 ? 1 : -1;
  const double sign = r.s > 0 ? 1.0 : -1.0;
  for (int i = 1; i <= nq; ++i) {
    const double t = __dadd_rn(__dmul_rn((double)i, r.base), r.offset);
    double f = floor(sign * t);
    f = f < -bound - 1.0 ? -bound - 1.0 : f;
    f = f > bound ? bound : f;
    o[i] = (int32_t)f;
  }
}

}  // namespace

hipError_t launch_expand_thresholds(const ifq_thr_compact* recs, int c_out, int out_bits,
                                    double bound, int32_t* thr, hipStream_t stream) {
  const int nq = (1 << out_bits) - 1;
  hipLaunchKernelGGL(expand_thresholds, dim3((c_out + 255) / 256), dim3(256), 0, stream, recs,
                     c_out, nq, bound, thr);
  return hipGetLastError();
}

}  // namespace ifq
