// Backward pass of the fused graph-transformer attention (included by
// gt_attn.hip inside its anonymous namespace; uses its device helpers, the
// degree partition kernel and the call workspace).
//
// Gradients for an upstream gradient dO (paper, Appendix D.2, backward pass of
// the graph transformer: the weights are recomputed from the stored per-row
// statistic L_i = ln sum_e exp(s_e), alpha_e = exp(s_e - L_i), and
// Delta_i = <O_i, dO_i>).  Per CSR entry e = (i, j) and head:
//     ds_e = alpha_e * (<dO_i, V_j> - Delta_i)
//     dQ_i += scale * ds_e * K_j          (pass 0, CSR rows i)
//     dK_j += scale * ds_e * Q_i          (pass 1, transposed rows j)
//     dV_j += alpha_e * dO_i              (pass 1)
// The paper's kernel walks the transposed graph and adds dK with atomics;
// here both passes are gathers over rows (the transposed structure is an
// input, as the paper's cached transposed adjacency), split rows are summed
// in chunk order, and the results are bitwise reproducible.
//
// Both passes have the same per-entry shape, with (a, b) the row's own
// vectors and (x, y) the gathered ones:
//     pass 0: a = Q_i, b = dO_i, x = K_j, y = V_j, (L, Delta) of the row i
//     pass 1: a = K_j, b = V_j, x = Q_i, y = dO_i, (L, Delta) gathered at i
//     s = <a, x> scale, alpha = exp(s - L), ds = alpha (<b, y> - Delta)
//     acc1 += ds x;  pass 1 also: acc2 += alpha y

struct BwdParams {
    const int64_t* rowptr;  // rows of this pass (CSR or transposed CSR)
    const int32_t* colidx;
    const char* A;  // row-own vectors a / b
    const char* B;
    const char* X;  // gathered vectors x / y
    const char* Y;
    const char* O;     // pass 0: forward output (for Delta)
    const float* lse;  // [N][H] natural log
    float* delta;      // [N][H]: written by pass 0, read by pass 1
    char* out1;        // dQ (pass 0) or dK (pass 1)
    char* out2;        // dV (pass 1)
    int64_t N;
    float c;      // scale * log2(e)
    float scale;
    int32_t light_max;
    int32_t cap_items;
    int32_t cap_heavy;
    const int32_t* counters;
    const int32_t* med_list;
    const ChunkItem* chunks;
    const HeavyRow* heavy;
    float* part;  // [slot][NACC * H * D]
};

// bf16 dot over the four pairs of two 16-byte vectors, accumulated in fp32
__device__ __forceinline__ float dot8_bf16(const uint4& a, const uint4& b) {
    float d = dot2_bf16(a.x, b.x, 0.0f);
    d = dot2_bf16(a.y, b.y, d);
    d = dot2_bf16(a.z, b.z, d);
    return dot2_bf16(a.w, b.w, d);
}

template <typename T, int H, int D, int MODE>
struct BwdState {
    using Gm = Geo<T, H, D>;
    static constexpr int NV = Gm::kNV, EPV = Gm::kEPV, U = Gm::kU;
    static constexpr int NACC = MODE ? 2 : 1;
    // bf16 features: the two dots per entry are bf16 dot2 on raw pairs, and
    // the accumulations pair two entries: their coefficients (ds, alpha) are
    // rounded to one bf16 pair and dot2 multiplies it with the two entries'
    // elements, accumulating in fp32.
    static constexpr bool kDot2 = std::is_same<T, bf16_tag>::value;
    static_assert(!kDot2 || U % 2 == 0, "dot2 pairs entries");
    float a[kDot2 ? 1 : NV][EPV], b[kDot2 ? 1 : NV][EPV];
    uint4 araw[kDot2 ? NV : 1], braw[kDot2 ? NV : 1];
    float acc1[NV][EPV], acc2[NV][EPV];
    float L2[NV], Dl[NV];  // pass 0: the row's statistics (per vector slot's head)

    __device__ __forceinline__ void begin(const BwdParams& p, int64_t row, int lig) {
        const int64_t off = row * (int64_t)Gm::kRowBytes + lig * 16;
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            const uint4 ar = *reinterpret_cast<const uint4*>(p.A + off + k * Gm::kG * 16);
            const uint4 br = *reinterpret_cast<const uint4*>(p.B + off + k * Gm::kG * 16);
            if constexpr (kDot2) {
                araw[k] = ar;
                braw[k] = br;
            } else {
                widen<T>(ar, a[k]);
                widen<T>(br, b[k]);
            }
#pragma unroll
            for (int e = 0; e < EPV; ++e) acc1[k][e] = acc2[k][e] = 0.0f;
        }
        if constexpr (MODE == 0) {
#pragma unroll
            for (int k = 0; k < NV; ++k) {
                const int v = lig + k * Gm::kG, h = v / Gm::kHL;
                const uint4 orw = *reinterpret_cast<const uint4*>(p.O + off + k * Gm::kG * 16);
                float d = 0.0f;
                if constexpr (kDot2) {
                    d = dot8_bf16(orw, braw[k]);
                } else {
                    float o[EPV];
                    widen<T>(orw, o);
#pragma unroll
                    for (int e = 0; e < EPV; ++e) d = fmaf(o[e], b[k][e], d);
                }
                Dl[k] = head_sum<Gm::kHL>(d);
                L2[k] = p.lse[row * H + h] * 1.4426950408889634f;
                if (v % Gm::kHL == 0) p.delta[row * H + h] = Dl[k];
            }
        }
    }

    __device__ __forceinline__ void step(const BwdParams& p, const int32_t (&j)[U], int nvalid, int lig) {
#pragma clang fp contract(off)
        uint4 xr[U][NV], yr[U][NV];
        float lg[U][NV], dg[U][NV];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t off = (int64_t)j[u] * Gm::kRowBytes + lig * 16;
#pragma unroll
            for (int k = 0; k < NV; ++k) {
                xr[u][k] = *reinterpret_cast<const uint4*>(p.X + off + k * Gm::kG * 16);
                yr[u][k] = *reinterpret_cast<const uint4*>(p.Y + off + k * Gm::kG * 16);
                if constexpr (MODE == 1) {
                    const int h = (lig + k * Gm::kG) / Gm::kHL;
                    lg[u][k] = p.lse[(int64_t)j[u] * H + h];
                    dg[u][k] = p.delta[(int64_t)j[u] * H + h];
                }
            }
        }
        if constexpr (kDot2) {
#pragma unroll
            for (int u = 0; u < U; u += 2) {
#pragma unroll
                for (int k = 0; k < NV; ++k) {
                    float al[2], ds[2];
#pragma unroll
                    for (int t = 0; t < 2; ++t) {
                        const float sc = head_sum<Gm::kHL>(dot8_bf16(araw[k], xr[u + t][k])) * p.c;
                        const float dd = head_sum<Gm::kHL>(dot8_bf16(braw[k], yr[u + t][k]));
                        const float l2 = MODE == 1 ? lg[u + t][k] * 1.4426950408889634f : L2[k];
                        const float dl = MODE == 1 ? dg[u + t][k] : Dl[k];
                        al[t] = (u + t < nvalid) ? fast_exp2(sc - l2) : 0.0f;
                        ds[t] = al[t] * (dd - dl);
                    }
                    const uint32_t pds = pack_bf16(ds[0], ds[1]);
                    const uint32_t pal = pack_bf16(al[0], al[1]);
                    const uint4 x0 = xr[u][k], x1 = xr[u + 1][k], y0 = yr[u][k], y1 = yr[u + 1][k];
                    const uint32_t xa[4] = {x0.x, x0.y, x0.z, x0.w}, xb[4] = {x1.x, x1.y, x1.z, x1.w};
                    const uint32_t ya[4] = {y0.x, y0.y, y0.z, y0.w}, yb[4] = {y1.x, y1.y, y1.z, y1.w};
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        acc1[k][2 * q] = dot2_bf16(pds, pair_lo(xa[q], xb[q]), acc1[k][2 * q]);
                        acc1[k][2 * q + 1] = dot2_bf16(pds, pair_hi(xa[q], xb[q]), acc1[k][2 * q + 1]);
                        if constexpr (MODE == 1) {
                            acc2[k][2 * q] = dot2_bf16(pal, pair_lo(ya[q], yb[q]), acc2[k][2 * q]);
                            acc2[k][2 * q + 1] = dot2_bf16(pal, pair_hi(ya[q], yb[q]), acc2[k][2 * q + 1]);
                        }
                    }
                }
            }
            return;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int k = 0; k < NV; ++k) {
                float x[EPV], y[EPV];
                widen<T>(xr[u][k], x);
                widen<T>(yr[u][k], y);
                float s = 0.0f, da = 0.0f;
#pragma unroll
                for (int e = 0; e < EPV; ++e) {
                    s = fmaf(a[k][e], x[e], s);
                    da = fmaf(b[k][e], y[e], da);
                }
                s = head_sum<Gm::kHL>(s) * p.c;
                da = head_sum<Gm::kHL>(da);
                const float l2 = MODE == 1 ? lg[u][k] * 1.4426950408889634f : L2[k];
                const float dl = MODE == 1 ? dg[u][k] : Dl[k];
                const float alpha = (u < nvalid) ? fast_exp2(s - l2) : 0.0f;
                const float ds = alpha * (da - dl);
#pragma unroll
                for (int e = 0; e < EPV; ++e) {
                    acc1[k][e] = fmaf(ds, x[e], acc1[k][e]);
                    if constexpr (MODE == 1) acc2[k][e] = fmaf(alpha, y[e], acc2[k][e]);
                }
            }
        }
    }

    __device__ __forceinline__ void sum_xor(int off) {
#pragma unroll
        for (int k = 0; k < NV; ++k)
#pragma unroll
            for (int e = 0; e < EPV; ++e) {
                acc1[k][e] += __shfl_xor(acc1[k][e], off);
                if constexpr (MODE == 1) acc2[k][e] += __shfl_xor(acc2[k][e], off);
            }
    }

    __device__ __forceinline__ void store(const BwdParams& p, int64_t row, int lig) const {
        const int64_t off = row * (int64_t)Gm::kRowBytes + lig * 16;
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            float o[EPV];
#pragma unroll
            for (int e = 0; e < EPV; ++e) o[e] = acc1[k][e] * p.scale;
            *reinterpret_cast<uint4*>(p.out1 + off + k * Gm::kG * 16) = narrow<T>(o);
            if constexpr (MODE == 1)
                *reinterpret_cast<uint4*>(p.out2 + off + k * Gm::kG * 16) = narrow<T>(acc2[k]);
        }
    }

    __device__ __forceinline__ void store_partial(const BwdParams& p, int32_t slot, int lig) const {
#pragma unroll
        for (int k = 0; k < NV; ++k) {
            const int v = lig + k * Gm::kG;
            float* dst = p.part + (int64_t)slot * NACC * Gm::kHD + v * EPV;
#pragma unroll
            for (int e = 0; e < EPV; e += 4) {
                *reinterpret_cast<float4*>(dst + e) = make_float4(acc1[k][e], acc1[k][e + 1], acc1[k][e + 2], acc1[k][e + 3]);
                if constexpr (MODE == 1)
                    *reinterpret_cast<float4*>(dst + Gm::kHD + e) =
                        make_float4(acc2[k][e], acc2[k][e + 1], acc2[k][e + 2], acc2[k][e + 3]);
            }
        }
    }
};

template <typename T, int H, int D, int MODE>
__device__ __forceinline__ void bwd_wave_segment(const BwdParams& p, int64_t row, int64_t b, int64_t e, int32_t slot,
                                                 int32_t* __restrict__ tile, int lane) {
    using Gm = Geo<T, H, D>;
    constexpr int U = Gm::kU, P = Gm::kP, G = Gm::kG;
    const int g = lane / G, lig = lane % G;
    BwdState<T, H, D, MODE> st;
    st.begin(p, row, lig);
    for (int64_t tb = b; tb < e; tb += kWave) {
        const int64_t pos = (tb + lane < e) ? tb + lane : e - 1;
        const int32_t idx = p.colidx[pos];
        wave_lds_fence();
        tile[lane] = idx;
        wave_lds_fence();
        const int nt = (int)((e - tb) < kWave ? (e - tb) : kWave);
        for (int t = 0; t < nt; t += P * U) {
            const int e0 = t + g * U;
            const int nvalid = nt - e0 < U ? nt - e0 : U;
            if (nvalid > 0) {
                int32_t j[U];
#pragma unroll
                for (int u = 0; u < U; ++u) j[u] = tile[e0 + u];
                st.step(p, j, nvalid, lig);
            }
        }
    }
#pragma unroll
    for (int off = G; off < kWave; off <<= 1) st.sum_xor(off);
    if (g == 0) {
        if (slot < 0)
            st.store(p, row, lig);
        else
            st.store_partial(p, slot, lig);
    }
}

template <typename T, int H, int D, int MODE>
__global__ void __launch_bounds__(kBlock) gt_bwd_kernel(BwdParams p) {
    using Gm = Geo<T, H, D>;
    constexpr int U = Gm::kU, G = Gm::kG;
    __shared__ int32_t tiles[kWavesPerBlock][kWave];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x / kWave;
    int32_t* tile = tiles[wv];
    const int32_t n_chunks = min(CNT(p.counters, CNT_CHUNKS), p.cap_items);
    const int32_t n_items = n_chunks + (int32_t)min((int64_t)CNT(p.counters, CNT_MED), p.N);
    const int nwaves = gridDim.x * kWavesPerBlock;
    for (int it = blockIdx.x * kWavesPerBlock + wv; it < n_items; it += nwaves) {
        if (it < n_chunks) {
            const ChunkItem ci = p.chunks[it];
            bwd_wave_segment<T, H, D, MODE>(p, ci.row, ci.begin, ci.end, ci.slot, tile, lane);
        } else {
            const int64_t row = p.med_list[it - n_chunks];
            bwd_wave_segment<T, H, D, MODE>(p, row, p.rowptr[row], p.rowptr[row + 1], -1, tile, lane);
        }
    }
    // light rows: one lane group each, P rows per wave
    const int g = lane / G, lig = lane % G;
    int32_t* gtile = tile + g * G;
    const int64_t n_light = (p.N + Gm::kP - 1) / Gm::kP;
    for (int64_t it = (int64_t)blockIdx.x * kWavesPerBlock + wv; it < n_light; it += nwaves) {
        const int64_t row = it * Gm::kP + g;
        if (row >= p.N) continue;
        const int64_t b = p.rowptr[row], e = p.rowptr[row + 1];
        if (e - b > p.light_max) continue;
        BwdState<T, H, D, MODE> st;
        st.begin(p, row, lig);
        for (int64_t tb = b; tb < e; tb += G) {
            const int32_t idx = p.colidx[(tb + lig < e) ? tb + lig : e - 1];
            wave_lds_fence();
            gtile[lig] = idx;
            wave_lds_fence();
            const int nt = (int)((e - tb) < G ? (e - tb) : G);
            for (int t = 0; t < nt; t += U) {
                const int nvalid = nt - t < U ? nt - t : U;
                int32_t j[U];
#pragma unroll
                for (int u = 0; u < U; ++u) j[u] = gtile[t + u];
                st.step(p, j, nvalid, lig);
            }
        }
        st.store(p, row, lig);
    }
}

// Ordered sum of the chunk partials of each split row, then scaling / storing.
template <typename T, int H, int D, int MODE>
__global__ void __launch_bounds__(kBlock) gt_bwd_merge_kernel(BwdParams p) {
    constexpr int HD = H * D;
    constexpr int NACC = MODE ? 2 : 1;
    constexpr int F = HD >= kWave ? HD / kWave : 1;
    constexpr int EB = Elt<T>::kBytes;
    const int lane = threadIdx.x & (kWave - 1);
    const int f0 = lane * F;
    const int32_t n_heavy = min(CNT(p.counters, CNT_HEAVY), p.cap_heavy);
    const int nwaves = gridDim.x * kWavesPerBlock;
    for (int hr = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; hr < n_heavy; hr += nwaves) {
        if (f0 >= HD) continue;
        const HeavyRow w = p.heavy[hr];
        float s1[F], s2[F];
#pragma unroll
        for (int f = 0; f < F; ++f) s1[f] = s2[f] = 0.0f;
        // a batch holds at most 64 partial floats per lane
        constexpr int kPer = (MODE ? 2 : 1) * F;
        constexpr int kB = 64 / kPer < kMergeBatch ? (64 / kPer > 1 ? 64 / kPer : 1) : kMergeBatch;
        for (int c0 = 0; c0 < w.nch; c0 += kB) {
            float a1[kB][F], a2[kB][F];
#pragma unroll
            for (int u = 0; u < kB; ++u) {
                const int64_t slot = w.base + (c0 + u < w.nch ? c0 + u : w.nch - 1);
                const float* src = p.part + slot * NACC * HD + f0;
#pragma unroll
                for (int f = 0; f < F; ++f) {
                    a1[u][f] = src[f];
                    a2[u][f] = MODE ? src[HD + f] : 0.0f;
                }
            }
            // chunks past the row's last add nothing (selects, not a loop exit,
            // so that the batch's loads stay ahead of their use)
#pragma unroll
            for (int u = 0; u < kB; ++u) {
                const bool valid = c0 + u < w.nch;
#pragma unroll
                for (int f = 0; f < F; ++f) {
                    const float t1 = s1[f] + a1[u][f], t2 = s2[f] + a2[u][f];
                    s1[f] = valid ? t1 : s1[f];
                    s2[f] = valid ? t2 : s2[f];
                }
            }
        }
        const int64_t base = (int64_t)w.row * HD + f0;
#pragma unroll
        for (int f = 0; f < F; ++f) {
            const float o1 = s1[f] * p.scale;
            if constexpr (EB == 4) {
                reinterpret_cast<float*>(p.out1)[base + f] = o1;
                if (MODE) reinterpret_cast<float*>(p.out2)[base + f] = s2[f];
            } else {
                reinterpret_cast<uint16_t*>(p.out1)[base + f] = (uint16_t)bf16_rne(o1);
                if (MODE) reinterpret_cast<uint16_t*>(p.out2)[base + f] = (uint16_t)bf16_rne(s2[f]);
            }
        }
    }
}

struct BwdArgs {
    const int64_t* rowptr;
    const int32_t* colidx;
    const int64_t* rowptr_t;
    const int32_t* colidx_t;
    const void* Q;
    const void* K;
    const void* V;
    const void* O;
    const void* dO;
    const float* lse;
    void* dQ;
    void* dK;
    void* dV;
    int64_t N, E;
    int32_t H, D;
    float scale;
};

template <typename T, int H, int D>
gt_status launch_bwd(const BwdArgs& a, hipStream_t stream) {
    using Gm = Geo<T, H, D>;
    const int light_max = 8 * Gm::kU;
    const int chunk = default_chunk_long(a.E, 2 * Gm::kRowBytes, Gm::kP * Gm::kU);  // both passes gather two rows
    const int heavy_min = default_front(chunk, Gm::kP);
    int dev = 0;
    if (const gt_status ds = call_device(stream, &dev); ds != GT_SUCCESS) return ds;
    hipError_t he = hipSuccess;
    const int64_t resident = (int64_t)device_cus(dev) * 4;
    const int64_t light_items = (a.N + Gm::kP - 1) / Gm::kP;
    int64_t g = light_items / (2 * kWavesPerBlock);
    if (g < 4 * resident) g = 4 * resident;
    if (g > 64 * resident) g = 64 * resident;
    const int64_t need = (light_items + kWavesPerBlock - 1) / kWavesPerBlock;
    if (g > need) g = need;
    const int grid = (int)(g > 0 ? g : 1);

    const PartCaps caps = part_caps(a.E, heavy_min, chunk);
    size_t off = 0;
    const size_t o_cnt = off;    off = align_up(off + 2 * kCntSetWords * sizeof(int32_t), 256);
    const size_t o_med = off;    off = align_up(off + (size_t)a.N * sizeof(int32_t), 256);
    const size_t o_heavy = off;  off = align_up(off + (size_t)caps.heavy * sizeof(HeavyRow), 256);
    const size_t o_chunks = off; off = align_up(off + (size_t)caps.items * sizeof(ChunkItem), 256);
    const size_t o_part = off;   off = align_up(off + (size_t)caps.slots * 2 * H * D * sizeof(float), 256);
    const size_t o_delta = off;  off = align_up(off + (size_t)a.N * H * sizeof(float), 256);
    const size_t ws_bytes = off;

    CallWorkspace cw;
    gt_status st = acquire_workspace(dev, ws_bytes, stream, cw);
    if (st != GT_SUCCESS) return st;
    char* ws = cw.ptr;
    int32_t* cnt_sets = reinterpret_cast<int32_t*>(ws + o_cnt);  // one counter set per pass
    if ((he = clear_counters(cnt_sets, 2 * kCntSetWords, stream)) != hipSuccess) return hip_fail(he, "counter clear");

    for (int mode = 0; mode < 2; ++mode) {
        int32_t* counters = cnt_sets + mode * kCntSetWords;
        const int64_t* rp = mode == 0 ? a.rowptr : a.rowptr_t;
        const int32_t* ci = mode == 0 ? a.colidx : a.colidx_t;

        PartParams pp;
        pp.rowptr = rp;
        pp.N = a.N;
        pp.light_max = light_max;
        pp.heavy_min = heavy_min;
        pp.chunk = chunk;
        pp.cap_heavy = (int32_t)caps.heavy;
        pp.cap_items = (int32_t)caps.items;
        pp.cap_slots = (int32_t)caps.slots;
        pp.counters = counters;
        pp.med_list = reinterpret_cast<int32_t*>(ws + o_med);
        pp.heavy = reinterpret_cast<HeavyRow*>(ws + o_heavy);
        pp.chunks = reinterpret_cast<ChunkItem*>(ws + o_chunks);
        if ((he = launch_partition(pp, stream)) != hipSuccess) return hip_fail(he, "partition launch");

        BwdParams bp;
        bp.rowptr = rp;
        bp.colidx = ci;
        bp.A = static_cast<const char*>(mode == 0 ? a.Q : a.K);
        bp.B = static_cast<const char*>(mode == 0 ? a.dO : a.V);
        bp.X = static_cast<const char*>(mode == 0 ? a.K : a.Q);
        bp.Y = static_cast<const char*>(mode == 0 ? a.V : a.dO);
        bp.O = static_cast<const char*>(a.O);
        bp.lse = a.lse;
        bp.delta = reinterpret_cast<float*>(ws + o_delta);
        bp.out1 = static_cast<char*>(mode == 0 ? a.dQ : a.dK);
        bp.out2 = static_cast<char*>(a.dV);
        bp.N = a.N;
        bp.c = a.scale * 1.4426950408889634f;
        bp.scale = a.scale;
        bp.light_max = light_max;
        bp.cap_items = (int32_t)caps.items;
        bp.cap_heavy = (int32_t)caps.heavy;
        bp.counters = counters;
        bp.med_list = pp.med_list;
        bp.chunks = pp.chunks;
        bp.heavy = pp.heavy;
        bp.part = reinterpret_cast<float*>(ws + o_part);
        int merge_grid = (int)((caps.heavy + kWavesPerBlock - 1) / kWavesPerBlock);
        if (merge_grid > device_cus(dev) * 8) merge_grid = device_cus(dev) * 8;
        if (merge_grid < 1) merge_grid = 1;
        if (mode == 0) {
            hipLaunchKernelGGL((gt_bwd_kernel<T, H, D, 0>), dim3(grid), dim3(kBlock), 0, stream, bp);
            if ((he = hipGetLastError()) != hipSuccess) return hip_fail(he, "backward launch");
            hipLaunchKernelGGL((gt_bwd_merge_kernel<T, H, D, 0>), dim3(merge_grid), dim3(kBlock), 0, stream, bp);
        } else {
            hipLaunchKernelGGL((gt_bwd_kernel<T, H, D, 1>), dim3(grid), dim3(kBlock), 0, stream, bp);
            if ((he = hipGetLastError()) != hipSuccess) return hip_fail(he, "backward launch");
            hipLaunchKernelGGL((gt_bwd_merge_kernel<T, H, D, 1>), dim3(merge_grid), dim3(kBlock), 0, stream, bp);
        }
        if ((he = hipGetLastError()) != hipSuccess) return hip_fail(he, "backward merge launch");
    }
    return GT_SUCCESS;
}

using BwdFn = gt_status (*)(const BwdArgs&, hipStream_t);

template <typename T>
BwdFn pick_bwd(int32_t H, int32_t D) {
#define GT_CASE(h, d) \
    if (H == h && D == d) return &launch_bwd<T, h, d>;
    GT_CASE(1, 32) GT_CASE(1, 64) GT_CASE(1, 128)
    GT_CASE(2, 32) GT_CASE(2, 64) GT_CASE(2, 128)
    GT_CASE(4, 32) GT_CASE(4, 64) GT_CASE(4, 128)
    GT_CASE(8, 32) GT_CASE(8, 64) GT_CASE(8, 128)
    GT_CASE(1, 256) GT_CASE(2, 256) GT_CASE(4, 256) GT_CASE(8, 256)
    if constexpr (std::is_same<T, bf16_tag>::value) {  // a head must fit 64 lanes of 16 bytes
        GT_CASE(1, 512) GT_CASE(2, 512) GT_CASE(4, 512)
    }
#undef GT_CASE
    return nullptr;
}
