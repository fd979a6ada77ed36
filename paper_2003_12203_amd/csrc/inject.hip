// Test-only fault injection into stored outputs (the paper corrupts selected
// output elements at source level, Sec. 6.1).  One thread applies the faults in
// list order, so repeated hits on one element compose deterministically.
#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

template <typename T>
__global__ void inject_kernel(T *O, Geom g, FaultList fl) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    for (int i = 0; i < fl.n; ++i) {
        const ftcnn_fault &f = fl.f[i];
        const long long idx = (((long long)f.n * g.M + f.m) * g.E + f.x) * g.F + f.y;
        O[idx] = fault_apply(O[idx], f);
    }
}

}  // namespace

hipError_t launch_inject(const Plan &pl, void *O, const ftcnn_fault *f, int nf, hipStream_t st) {
    FaultList fl;
    for (int i = 0; i < nf; ++i) fl.f[i] = f[i];
    fl.n = nf;
    if (pl.g.dtype == FTCNN_F32)
        inject_kernel<float><<<1, 64, 0, st>>>(static_cast<float *>(O), pl.g, fl);
    else
        inject_kernel<uint16_t><<<1, 64, 0, st>>>(static_cast<uint16_t *>(O), pl.g, fl);
    return hipGetLastError();
}

}  // namespace ftcnn
