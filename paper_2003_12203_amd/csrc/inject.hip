// Test-only fault injection into stored outputs (the paper corrupts selected
// output elements at source level, Sec. 6.1).  One thread applies the faults in
// list order, so repeated hits on one element compose deterministically.
#include "ftcnn_internal.h"

namespace ftcnn {
namespace {

struct FaultList {
    ftcnn_fault f[kMaxFaults];
    int n;
};

template <typename T>
__global__ void inject_kernel(T *O, Geom g, FaultList fl) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    for (int i = 0; i < fl.n; ++i) {
        const ftcnn_fault &f = fl.f[i];
        const long long idx = (((long long)f.n * g.M + f.m) * g.E + f.x) * g.F + f.y;
        if (f.kind == 0) {
            if constexpr (sizeof(T) == 4) {
                const uint32_t b = __builtin_bit_cast(uint32_t, O[idx]) ^ (1u << f.bit);
                O[idx] = __builtin_bit_cast(float, b);
            } else {
                O[idx] = (T)(O[idx] ^ (uint16_t)(1u << f.bit));
            }
        } else {
            const double old = (double)Elem<T>::load(O, idx);
            const double v = f.kind == 1 ? old + f.value : f.value;
            Elem<T>::store(O, idx, (float)v);
        }
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
