// Locality microbenchmark of the reordering study (paper: graph reordering
// paragraph of Section 4 and the appendix figure of the reordering gap).  A
// "dot-aggr" kernel with identical arithmetic under two wave-per-node
// mappings, so that only the memory access pattern differs:
//     s[i] = sum over the CSR entries e of row i of <X[i,:], X[j_e,:]>
//   * feature-parallel (MAP 0): the wave's lanes own consecutive features of
//     the row; neighbours are scanned one after another (four in flight), so
//     every load instruction reads one contiguous piece of one neighbour row;
//   * neighbour-parallel (MAP 1): lane l takes entries l, l+64, ... and reads
//     its neighbour's whole row itself (x_i staged in LDS), so one load
//     instruction touches 64 different rows and relies on cache reuse.
// VB is the bytes per lane per load: 4 (scalar) or 16 (vectorised).
// Accumulation is fp32 per lane, then a tree over the wave.  The study times
// these kernels on the original and on relabeled graphs.
// This file is included by gt_attn.hip inside its anonymous namespace.

struct DotParams {
    const int64_t* rowptr;
    const int32_t* colidx;
    const float* X;
    float* out;
    int64_t N;
};

template <int VB> __device__ __forceinline__ void load_floats(const float* __restrict__ src, float* dst) {
    if constexpr (VB == 16) {
        const float4 v = *reinterpret_cast<const float4*>(src);
        dst[0] = v.x;
        dst[1] = v.y;
        dst[2] = v.z;
        dst[3] = v.w;
    } else {
        dst[0] = *src;
    }
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

template <int MAP, int VB, int F>
__global__ void __launch_bounds__(kBlock) gt_dot_aggr_kernel(DotParams p) {
    constexpr int EPL = VB / 4;                       // floats per load
    constexpr int NVEC = F / EPL;                      // loads per row
    __shared__ float xs[kWavesPerBlock][MAP == 1 ? F : 1];
    const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
    const int64_t row = (int64_t)blockIdx.x * kWavesPerBlock + wv;
    if (row >= p.N) return;  // a whole wave leaves together; no block barrier follows
    const int64_t b = p.rowptr[row], e = p.rowptr[row + 1];
    const float* xi = p.X + row * F;
    float acc = 0.0f;
    if constexpr (MAP == 0) {
        // lane owns loads v = lane + 64 k (k < NL); lanes past NVEC are idle
        constexpr int NL = NVEC > kWave ? NVEC / kWave : 1;
        const bool active = lane < NVEC;
        float q[NL][EPL];
#pragma unroll
        for (int k = 0; k < NL; ++k) {
            if (active) {
                load_floats<VB>(xi + (lane + k * kWave) * EPL, q[k]);
            } else {
#pragma unroll
                for (int t = 0; t < EPL; ++t) q[k][t] = 0.0f;
            }
        }
        constexpr int UN = 4;
        for (int64_t t0 = b; t0 < e; t0 += UN) {
            float x[UN][NL][EPL];
#pragma unroll
            for (int u = 0; u < UN; ++u) {
                const int64_t t = t0 + u < e ? t0 + u : e - 1;
                const float* xj = p.X + (int64_t)p.colidx[t] * F;
#pragma unroll
                for (int k = 0; k < NL; ++k) {
                    if (active) {
                        load_floats<VB>(xj + (lane + k * kWave) * EPL, x[u][k]);
                    } else {
#pragma unroll
                        for (int c = 0; c < EPL; ++c) x[u][k][c] = 0.0f;
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < UN; ++u) {
                if (t0 + u < e) {
#pragma unroll
                    for (int k = 0; k < NL; ++k)
#pragma unroll
                        for (int c = 0; c < EPL; ++c) acc = fmaf(q[k][c], x[u][k][c], acc);
                }
            }
        }
    } else {
        // stage x_i in LDS (one coalesced pass), then each lane walks its own
        // neighbours' rows against the broadcast copy
        for (int f = lane; f < F; f += kWave) xs[wv][f] = xi[f];
        wave_lds_fence();
        for (int64_t t = b + lane; t < e; t += kWave) {
            const float* xj = p.X + (int64_t)p.colidx[t] * F;
#pragma unroll 8
            for (int v = 0; v < NVEC; ++v) {
                float x[EPL];
                load_floats<VB>(xj + v * EPL, x);
#pragma unroll
                for (int c = 0; c < EPL; ++c) acc = fmaf(xs[wv][v * EPL + c], x[c], acc);
            }
        }
    }
    acc = wave_sum(acc);
    if (lane == 0) p.out[row] = acc;
}

using DotFn = void (*)(DotParams);

template <int MAP, int VB>
DotFn pick_dot_f(int32_t F) {
    switch (F) {
        case 32: return &gt_dot_aggr_kernel<MAP, VB, 32>;
        case 64: return &gt_dot_aggr_kernel<MAP, VB, 64>;
        case 128: return &gt_dot_aggr_kernel<MAP, VB, 128>;
        case 256: return &gt_dot_aggr_kernel<MAP, VB, 256>;
        case 512: return &gt_dot_aggr_kernel<MAP, VB, 512>;
        default: return nullptr;
    }
}

DotFn pick_dot(int32_t mapping, int32_t load_bytes, int32_t F) {
    if (mapping == 0) return load_bytes == 16 ? pick_dot_f<0, 16>(F) : load_bytes == 4 ? pick_dot_f<0, 4>(F) : nullptr;
    if (mapping == 1) return load_bytes == 16 ? pick_dot_f<1, 16>(F) : load_bytes == 4 ? pick_dot_f<1, 4>(F) : nullptr;
    return nullptr;
}
