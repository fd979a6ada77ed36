// One workgroup's share of the input checksums Cd1 = sum_n D_n and
// Cd2 = sum_n (n + wbase) D_n (Sec. 3.2), for workgroups that run it beside
// other work in the same launch (the convolution's, or the channels-last
// rearrangement's).  Device code shared by those launches.
#pragma once

#include <type_traits>

#include "ftcnn_internal.h"

namespace ftcnn {

constexpr int kEncVec = 4;   // columns per thread in the encode workgroups

// V elements of one row of D, loaded as one unit (V * sizeof(T) is 2 to 16 bytes).
template <typename T, int V> union RowPack {
    using Q = typename std::conditional<
        V * sizeof(T) == 16, uint4,
        typename std::conditional<V * sizeof(T) == 8, uint2,
                                  typename std::conditional<V * sizeof(T) == 4, uint32_t, uint16_t>::type>::type>::type;
    Q q;
    T e[V];
};

// One encode workgroup: V consecutive columns of D viewed as [N][Ch*H*W] per
// thread, every row n in order (eight rows of loads in flight), accumulated in
// float64: Cd1 = sum_n D_n and Cd2 = sum_n (n + wbase) D_n.
template <typename T, int NT, int V>
__device__ inline void encode_block(const T *__restrict__ D, const Geom &g, int blk, double *__restrict__ cd1,
                             double *__restrict__ cd2) {
    const long long col = ((long long)blk * NT + threadIdx.x) * V;
    if (col >= g.CHW) return;
    const int nv = (long long)V <= g.CHW - col ? V : (int)(g.CHW - col);   // V == 1 whenever Ch*H*W % V != 0
    double a1[V], a2[V];
#pragma unroll
    for (int e = 0; e < V; ++e) a1[e] = a2[e] = 0.0;
    const T *src = D + col;
    // rows stay packed in registers until they are added (V elements per row in flight)
    using P = RowPack<T, V>;
    auto load = [&](long long row) -> P {
        P pk;
        pk.q = *reinterpret_cast<const typename P::Q *>(src + row * g.CHW);
        return pk;
    };
    auto add = [&](const P &pk, int n) {
        const double w = (double)(n + g.wbase);
#pragma unroll
        for (int e = 0; e < V; ++e) {
            double x;
            if constexpr (sizeof(T) == 4) x = (double)pk.e[e];
            else x = (double)bf16_bits_to_f32(pk.e[e]);
            a1[e] += x;
            a2[e] = fma(w, x, a2[e]);
        }
    };
    int n = 0;
    for (; n + 7 < g.N; n += 8) {
        P v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = load(n + u);
#pragma unroll
        for (int u = 0; u < 8; ++u) add(v[u], n + u);
    }
    for (; n < g.N; ++n) add(load(n), n);
#pragma unroll
    for (int e = 0; e < V; ++e)
        if (e < nv) {
            cd1[col + e] = a1[e];
            cd2[col + e] = a2[e];
        }
}

}  // namespace ftcnn
