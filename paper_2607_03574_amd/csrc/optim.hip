// Adam update of a population of parameter vectors (the calibration loop
// that drives the gradient replay: an optimiser fits each lane's parameters
// against the observations with exact gradients, Section "From buckets to
// phases", the Kalman maximum-likelihood fit).  Adam as published by Kingma
// and Ba (2015), with bias correction:
//   m <- b1 m + (1 - b1) g,  v <- b2 v + (1 - b2) g g,
//   p <- p - lr (m / c1) / (sqrt(v / c2) + eps),  c1 = 1 - b1^t, c2 = 1 - b2^t.
// Elementwise and HBM bound (7 doubles of traffic per element): one thread
// per (lane, parameter), consecutive threads on consecutive parameters of a
// lane so each wave reads contiguous rows.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace ndvm {

struct AdamArgs {
    double *p;
    const double *g;
    double *m, *v;
    int64_t L, P, ld_p, ld_g;
    double lr, b1, b2, eps, c1, c2;
};

__global__ void __launch_bounds__(256) ndvm_adam(AdamArgs a) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= a.L * a.P) return;
    const int64_t l = i / a.P, k = i % a.P;
    const double g = a.g[l * a.ld_g + k];
    const double m = a.b1 * a.m[i] + (1.0 - a.b1) * g;
    const double v = a.b2 * a.v[i] + (1.0 - a.b2) * (g * g);
    a.m[i] = m;
    a.v[i] = v;
    const double mh = m / a.c1, vh = v / a.c2;
    double *p = a.p + l * a.ld_p + k;
    *p = *p - a.lr * mh / (sqrt(vh) + a.eps);
}

hipError_t launch_adam(const AdamArgs &a, hipStream_t stream) {
    const int64_t n = a.L * a.P;
    if (n == 0) return hipSuccess;
    const uint32_t blocks = uint32_t((n + 255) / 256);
    hipLaunchKernelGGL(ndvm_adam, dim3(blocks), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace ndvm
