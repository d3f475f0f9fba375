// Segment min/max aggregation over a CSR graph (the paper's reduction family,
// Section 2.2 family (ii); Appendix, degree-aware reduction-based
// aggregation).  For every destination row i and feature f:
//     out[i,f] = REDUCE over the CSR entries e of row i of X[j_e, f]
//     arg[i,f] = the source j_e that attains it (-1 for an empty row)
// with REDUCE = min or max under the order-preserving key of the paper's
// packed (value, index) merge: the fp32 bit pattern with all bits inverted
// when the sign bit is set and the sign bit set otherwise, compared as an
// unsigned integer, ties to the smallest source index.
//
// Design: each lane keeps, per feature it owns, one 64-bit word
// (key << 32 | source); the reduction is a plain unsigned 64-bit minimum
// (max uses the complemented key, so ties still go to the smallest source).
// The words are exactly the paper's packed atomics operands, but here they
// stay in registers: rows are mapped like the attention forward (one lane
// group per light row with 16-byte loads, one wave per medium row, chunks of
// long rows on different waves) and the chunk partials of long rows are
// merged by a second kernel instead of 64-bit atomics.  Padding entries of a
// step repeat a valid entry, which a minimum absorbs, so they need no mask.
// This file is included by gt_attn.hip inside its anonymous namespace.

template <typename T, int NVEC>
struct RedGeo {
    static constexpr int kEB = Elt<T>::kBytes;
    static constexpr int kEPV = 16 / kEB;  // elements per 16-byte vector
    static constexpr int kF = NVEC * kEPV;   // features per row
    static constexpr int kRowBytes = NVEC * 16;
    static constexpr int kG = NVEC < kWave ? NVEC : kWave;  // lanes per group
    static constexpr int kNV = NVEC / kG;                   // vectors per lane
    static constexpr int kP = kWave / kG;                   // groups per wave
    static constexpr int kU0 = (8 / kNV) > 2 ? (8 / kNV) : 2;
    static constexpr int kU = kU0 < kG ? kU0 : kG;          // entries per step
    static_assert(kG % kU == 0 && kP * kU <= kWave, "index tiles must cover whole steps");
};

struct ReduceParams {
    const int64_t* rowptr;
    const int32_t* colidx;
    const char* X;
    char* out;
    int32_t* arg;     // [N][F] or nullptr
    uint64_t* part;   // [slot][F] packed (key, source) of chunk partials
    int64_t N;
    uint32_t flip;    // 0 for min, 0xFFFFFFFF for max
    int32_t light_max;
    int32_t cap_items;
    int32_t cap_heavy;
    const int32_t* counters;
    const int32_t* med_list;
    const ChunkItem* chunks;
    const HeavyRow* heavy;
};

constexpr uint64_t kRedEmpty = ~0ull;  // no entry yet: source 0xFFFFFFFF is never valid

// Key of one fp32 bit pattern, complemented for max: bits ^ 0x80000000 for a
// clear sign bit, ~bits for a set one (then ^ flip).
__device__ __forceinline__ uint32_t red_key(uint32_t bits, uint32_t flip) {
    const uint32_t neg = (uint32_t)((int32_t)bits >> 31);
    return bits ^ (neg & 0x7FFFFFFFu) ^ (0x80000000u ^ flip);
}

// Inverse of red_key for the stored word: the fp32 bit pattern.
__device__ __forceinline__ uint32_t red_value_bits(uint64_t w, uint32_t flip) {
    const uint32_t k = (uint32_t)(w >> 32) ^ flip;
    return (k & 0x80000000u) ? (k ^ 0x80000000u) : ~k;
}

template <typename T> __device__ __forceinline__ uint32_t red_bits(const uint4& r, int e);
template <> __device__ __forceinline__ uint32_t red_bits<float>(const uint4& r, int e) {
    return e == 0 ? r.x : e == 1 ? r.y : e == 2 ? r.z : r.w;
}
template <> __device__ __forceinline__ uint32_t red_bits<bf16_tag>(const uint4& r, int e) {
    const uint32_t w = (e >> 1) == 0 ? r.x : (e >> 1) == 1 ? r.y : (e >> 1) == 2 ? r.z : r.w;
    return (e & 1) ? (w & 0xFFFF0000u) : (w << 16);
}

template <typename T, int NVEC>
struct RedState {
    using Gm = RedGeo<T, NVEC>;
    uint64_t best[Gm::kNV][Gm::kEPV];

    __device__ __forceinline__ void begin() {
#pragma unroll
        for (int k = 0; k < Gm::kNV; ++k)
#pragma unroll
            for (int e = 0; e < Gm::kEPV; ++e) best[k][e] = kRedEmpty;
    }

    struct Batch {
        uint4 x[Gm::kU][Gm::kNV];
    };

    __device__ __forceinline__ void issue(const char* __restrict__ Xb, const int32_t (&j)[Gm::kU], int lig,
                                          Batch& bt) const {
#pragma unroll
        for (int u = 0; u < Gm::kU; ++u) {
            const char* src = Xb + (int64_t)j[u] * Gm::kRowBytes + lig * 16;
#pragma unroll
            for (int k = 0; k < Gm::kNV; ++k) bt.x[u][k] = *reinterpret_cast<const uint4*>(src + k * Gm::kG * 16);
        }
    }

    __device__ __forceinline__ void consume(const Batch& bt, const int32_t (&j)[Gm::kU], uint32_t flip) {
#pragma unroll
        for (int u = 0; u < Gm::kU; ++u) {
#pragma unroll
            for (int k = 0; k < Gm::kNV; ++k) {
#pragma unroll
                for (int e = 0; e < Gm::kEPV; ++e) {
                    const uint64_t w = ((uint64_t)red_key(red_bits<T>(bt.x[u][k], e), flip) << 32) | (uint32_t)j[u];
                    best[k][e] = w < best[k][e] ? w : best[k][e];
                }
            }
        }
    }

    __device__ __forceinline__ void step(const char* __restrict__ Xb, const int32_t (&j)[Gm::kU], int lig,
                                         uint32_t flip) {
        Batch bt;
        issue(Xb, j, lig, bt);
        consume(bt, j, flip);
    }

    __device__ __forceinline__ void merge_xor(int off) {
#pragma unroll
        for (int k = 0; k < Gm::kNV; ++k)
#pragma unroll
            for (int e = 0; e < Gm::kEPV; ++e) {
                const uint32_t lo = __shfl_xor((uint32_t)best[k][e], off);
                const uint32_t hi = __shfl_xor((uint32_t)(best[k][e] >> 32), off);
                const uint64_t o = ((uint64_t)hi << 32) | lo;
                best[k][e] = o < best[k][e] ? o : best[k][e];
            }
    }

    __device__ __forceinline__ void store_out(const ReduceParams& p, int64_t row, int lig) const {
        char* orow = p.out + row * (int64_t)Gm::kRowBytes + lig * 16;
#pragma unroll
        for (int k = 0; k < Gm::kNV; ++k) {
            uint32_t vb[Gm::kEPV];
            int32_t src[Gm::kEPV];
#pragma unroll
            for (int e = 0; e < Gm::kEPV; ++e) {
                const bool none = (uint32_t)best[k][e] == 0xFFFFFFFFu;
                vb[e] = none ? 0u : red_value_bits(best[k][e], p.flip);
                src[e] = none ? -1 : (int32_t)(uint32_t)best[k][e];
            }
            uint4 o;
            if constexpr (Gm::kEB == 4) {
                o = make_uint4(vb[0], vb[1], vb[2], vb[3]);
            } else {
                // the selected value came from a bf16, so its low half is zero
                o = make_uint4((vb[0] >> 16) | (vb[1] & 0xFFFF0000u), (vb[2] >> 16) | (vb[3] & 0xFFFF0000u),
                               (vb[4] >> 16) | (vb[5] & 0xFFFF0000u), (vb[6] >> 16) | (vb[7] & 0xFFFF0000u));
            }
            *reinterpret_cast<uint4*>(orow + k * Gm::kG * 16) = o;
            if (p.arg) {
                int32_t* arow = p.arg + row * (int64_t)Gm::kF + (int64_t)(lig + k * Gm::kG) * Gm::kEPV;
#pragma unroll
                for (int e = 0; e < Gm::kEPV; e += 4)
                    *reinterpret_cast<int4*>(arow + e) = make_int4(src[e], src[e + 1], src[e + 2], src[e + 3]);
            }
        }
    }

    __device__ __forceinline__ void store_partial(uint64_t* __restrict__ part, int32_t slot, int lig) const {
#pragma unroll
        for (int k = 0; k < Gm::kNV; ++k) {
            uint64_t* dst = part + (int64_t)slot * Gm::kF + (int64_t)(lig + k * Gm::kG) * Gm::kEPV;
#pragma unroll
            for (int e = 0; e < Gm::kEPV; e += 2) {
                const uint64_t a = best[k][e], b = best[k][e + 1];
                *reinterpret_cast<uint4*>(dst + e) =
                    make_uint4((uint32_t)a, (uint32_t)(a >> 32), (uint32_t)b, (uint32_t)(b >> 32));
            }
        }
    }
};

// One wavefront over CSR entries [b, e) of `row`: the P groups take
// interleaved steps and are merged across lanes; slot < 0 writes the output,
// slot >= 0 the chunk partial.
template <typename T, int NVEC>
__device__ __forceinline__ void red_wave_segment(const ReduceParams& p, int64_t row, int64_t b, int64_t e,
                                                 int32_t slot, int32_t* __restrict__ tile, int lane) {
    using Gm = RedGeo<T, NVEC>;
    constexpr int U = Gm::kU, P = Gm::kP, G = Gm::kG;
    const int g = lane / G, lig = lane % G;
    RedState<T, NVEC> st;
    st.begin();
    for (int64_t tb = b; tb < e; tb += kWave) {
        const int64_t pos = (tb + lane < e) ? tb + lane : e - 1;
        const int32_t idx = p.colidx[pos];
        wave_lds_fence();
        tile[lane] = idx;
        wave_lds_fence();
        const int nt = (int)((e - tb) < kWave ? (e - tb) : kWave);
        for (int t = 0; t < nt; t += P * U) {
            const int e0 = t + g * U;
            if (e0 < nt) {
                int32_t j[U];
#pragma unroll
                for (int u = 0; u < U; ++u) j[u] = tile[e0 + u < nt ? e0 + u : nt - 1];
                st.step(p.X, j, lig, p.flip);
            }
        }
    }
#pragma unroll
    for (int off = G; off < kWave; off <<= 1) st.merge_xor(off);
    if (g == 0) {
        if (slot < 0)
            st.store_out(p, row, lig);
        else
            st.store_partial(p.part, slot, lig);
    }
}

// Light rows, one lane group each, software-pipelined across rows as in the
// attention forward: the next row's rowptr pair is loaded before the current
// row starts and its first index tile while the current row's first batch is
// in flight.
template <typename T, int NVEC>
__device__ __forceinline__ void red_light_rows(const ReduceParams& p, int64_t it, int64_t it_end, int64_t stride,
                                               int g, int lig, int32_t* __restrict__ gtile) {
    using Gm = RedGeo<T, NVEC>;
    constexpr int U = Gm::kU, G = Gm::kG, P = Gm::kP;
    int64_t row = it * P + g;
    bool ok = it < it_end && row < p.N;
    int64_t b = ok ? p.rowptr[row] : 0, e = ok ? p.rowptr[row + 1] : 0;
    bool mine = ok && (e - b) <= p.light_max;
    int32_t idx = (mine && e > b) ? p.colidx[(b + lig < e) ? b + lig : e - 1] : 0;
    while (it < it_end) {
        const int64_t crow = row, cb = b, ce = e;
        const bool cmine = mine;
        const int32_t cidx = idx;
        it += stride;
        row = it * P + g;
        ok = it < it_end && row < p.N;
        b = ok ? p.rowptr[row] : 0;
        e = ok ? p.rowptr[row + 1] : 0;
        mine = ok && (e - b) <= p.light_max;
        bool fetched = false;
        if (cmine) {
            RedState<T, NVEC> st;
            st.begin();
            for (int64_t tb = cb; tb < ce; tb += G) {
                int32_t tile_idx = cidx;
                if (tb != cb) tile_idx = p.colidx[(tb + lig < ce) ? tb + lig : ce - 1];
                wave_lds_fence();
                gtile[lig] = tile_idx;
                wave_lds_fence();
                const int nt = (int)((ce - tb) < G ? (ce - tb) : G);
                for (int t = 0; t < nt; t += U) {
                    int32_t j[U];
#pragma unroll
                    for (int u = 0; u < U; ++u) j[u] = gtile[t + u];
                    typename RedState<T, NVEC>::Batch bt;
                    st.issue(p.X, j, lig, bt);
                    if (!fetched) {
                        idx = (mine && e > b) ? p.colidx[(b + lig < e) ? b + lig : e - 1] : 0;
                        fetched = true;
                    }
                    st.consume(bt, j, p.flip);
                }
            }
            st.store_out(p, crow, lig);
        }
        if (!fetched) idx = (mine && e > b) ? p.colidx[(b + lig < e) ? b + lig : e - 1] : 0;
    }
}

template <typename T, int NVEC>
__global__ void __launch_bounds__(kBlock) gt_reduce_kernel(ReduceParams p) {
    using Gm = RedGeo<T, NVEC>;
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
            red_wave_segment<T, NVEC>(p, ci.row, ci.begin, ci.end, ci.slot, tile, lane);
        } else {
            const int64_t row = p.med_list[it - n_chunks];
            red_wave_segment<T, NVEC>(p, row, p.rowptr[row], p.rowptr[row + 1], -1, tile, lane);
        }
    }

    const int xcd = blockIdx.x % kXcds;
    const int waves_per_xcd = (gridDim.x / kXcds) * kWavesPerBlock;
    const int lw = (blockIdx.x / kXcds) * kWavesPerBlock + wv;
    const int64_t n_light = (p.N + Gm::kP - 1) / Gm::kP;
    const int64_t lo = n_light * xcd / kXcds, hi = n_light * (xcd + 1) / kXcds;
    const int g = lane / Gm::kG, lig = lane % Gm::kG;
    red_light_rows<T, NVEC>(p, lo + lw, hi, waves_per_xcd, g, lig, tile + g * Gm::kG);
}

// Merge of the chunk partials of each split row (one wave per row; lane l
// owns features l, l+64, ... so every load and store is coalesced).
template <typename T, int NVEC>
__global__ void __launch_bounds__(kBlock) gt_reduce_merge_kernel(ReduceParams p) {
    using Gm = RedGeo<T, NVEC>;
    constexpr int F = Gm::kF;
    constexpr int PER = (F + kWave - 1) / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    const int32_t n_heavy = min(CNT(p.counters, CNT_HEAVY), p.cap_heavy);
    const int nwaves = gridDim.x * kWavesPerBlock;
    for (int hr = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; hr < n_heavy; hr += nwaves) {
        const HeavyRow w = p.heavy[hr];
        uint64_t best[PER];
#pragma unroll
        for (int q = 0; q < PER; ++q) best[q] = kRedEmpty;
        // kRB chunks per round (about 8 loads per lane in flight), loaded
        // before any is compared; a round past the row's last chunk re-reads
        // the last one, which leaves the minimum unchanged
        constexpr int kRB = 8 / PER > 1 ? 8 / PER : 1;
        for (int c0 = 0; c0 < w.nch; c0 += kRB) {
            uint64_t v[kRB][PER];
#pragma unroll
            for (int u = 0; u < kRB; ++u) {
                const int c = c0 + u < w.nch ? c0 + u : w.nch - 1;
                const uint64_t* src = p.part + (int64_t)(w.base + c) * F;
#pragma unroll
                for (int q = 0; q < PER; ++q) {
                    const int f = lane + q * kWave;
                    v[u][q] = f < F ? src[f] : kRedEmpty;
                }
            }
#pragma unroll
            for (int u = 0; u < kRB; ++u)
#pragma unroll
                for (int q = 0; q < PER; ++q) best[q] = v[u][q] < best[q] ? v[u][q] : best[q];
        }
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int f = lane + q * kWave;
            if (f >= F) continue;
            const bool none = (uint32_t)best[q] == 0xFFFFFFFFu;
            const uint32_t vb = none ? 0u : red_value_bits(best[q], p.flip);
            const int64_t o = (int64_t)w.row * F + f;
            if constexpr (Gm::kEB == 4)
                reinterpret_cast<uint32_t*>(p.out)[o] = vb;
            else
                reinterpret_cast<uint16_t*>(p.out)[o] = (uint16_t)(vb >> 16);
            if (p.arg) p.arg[o] = none ? -1 : (int32_t)(uint32_t)best[q];
        }
    }
}

struct ReduceArgs {
    const int64_t* rowptr;
    const int32_t* colidx;
    const void* X;
    void* out;
    int32_t* arg;
    int64_t N, E;
    int32_t F;
    uint32_t flip;
};

template <typename T, int NVEC>
int reduce_blocks_per_cu(int dev) {
    static std::atomic<int> cache[64];
    if (dev < 0 || dev >= 64) return 4;
    if (cache[dev] == 0) {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, gt_reduce_kernel<T, NVEC>, kBlock, 0) != hipSuccess ||
            nb <= 0)
            nb = 4;
        cache[dev] = nb;
    }
    return cache[dev];
}

template <typename T, int NVEC>
gt_status launch_reduce(const ReduceArgs& a, const gt_tuning* tu, hipStream_t stream) {
    using Gm = RedGeo<T, NVEC>;
    int light_max = 8 * Gm::kU;
    int chunk = default_chunk_long(a.E, Gm::kRowBytes, Gm::kP * Gm::kU);
    int heavy_min = default_front(chunk, Gm::kP);
    int grid = 0;
    if (tu) {
        if (tu->light_max_deg > 0) light_max = tu->light_max_deg;
        if (tu->heavy_min_deg > 0) heavy_min = tu->heavy_min_deg;
        if (tu->chunk_edges > 0) chunk = (tu->chunk_edges + kWave - 1) / kWave * kWave;
        if (tu->grid_blocks > 0) grid = tu->grid_blocks;
    }
    if (heavy_min <= light_max) heavy_min = light_max + 1;

    int dev = 0;
    if (const gt_status ds = call_device(stream, &dev); ds != GT_SUCCESS) return ds;
    hipError_t he = hipSuccess;
    if (grid <= 0) {
        const int64_t resident = (int64_t)device_cus(dev) * reduce_blocks_per_cu<T, NVEC>(dev);
        const int64_t light_items = (a.N + Gm::kP - 1) / Gm::kP;
        int64_t g = light_items / (2 * kWavesPerBlock);
        if (g < 4 * resident) g = 4 * resident;
        if (g > 64 * resident) g = 64 * resident;
        const int64_t need = (light_items + kWavesPerBlock - 1) / kWavesPerBlock;
        if (g > need) g = need;
        grid = (int)(g > 0 ? g : 1);
    }
    grid = (grid + kXcds - 1) / kXcds * kXcds;

    // workspace: counters | medium rows | split rows | chunk items | partials
    const PartCaps caps = part_caps(a.E, heavy_min, chunk);
    size_t off = 0;
    const size_t o_cnt = off;    off = align_up(off + kCntSetWords * sizeof(int32_t), 256);
    const size_t o_med = off;    off = align_up(off + (size_t)a.N * sizeof(int32_t), 256);
    const size_t o_heavy = off;  off = align_up(off + (size_t)caps.heavy * sizeof(HeavyRow), 256);
    const size_t o_chunks = off; off = align_up(off + (size_t)caps.items * sizeof(ChunkItem), 256);
    const size_t o_part = off;   off = align_up(off + (size_t)caps.slots * Gm::kF * sizeof(uint64_t), 256);
    const size_t ws_bytes = off;

    CallWorkspace cw;
    gt_status st = acquire_workspace(dev, ws_bytes, stream, cw);
    if (st != GT_SUCCESS) return st;
    char* ws = cw.ptr;
    int32_t* counters = reinterpret_cast<int32_t*>(ws + o_cnt);

    PhaseEvents ph;
    if ((he = ph.start(stream)) != hipSuccess) return hip_fail(he, "profiling events");
    if ((he = clear_counters(counters, kCntSetWords, stream)) != hipSuccess) return hip_fail(he, "counter clear");

    PartParams pp;
    pp.rowptr = a.rowptr;
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
    ph.mark(1, stream);

    ReduceParams rp;
    rp.rowptr = a.rowptr;
    rp.colidx = a.colidx;
    rp.X = static_cast<const char*>(a.X);
    rp.out = static_cast<char*>(a.out);
    rp.arg = a.arg;
    rp.part = reinterpret_cast<uint64_t*>(ws + o_part);
    rp.N = a.N;
    rp.flip = a.flip;
    rp.light_max = light_max;
    rp.cap_items = (int32_t)caps.items;
    rp.cap_heavy = (int32_t)caps.heavy;
    rp.counters = counters;
    rp.med_list = pp.med_list;
    rp.chunks = pp.chunks;
    rp.heavy = pp.heavy;
    hipLaunchKernelGGL((gt_reduce_kernel<T, NVEC>), dim3(grid), dim3(kBlock), 0, stream, rp);
    if ((he = hipGetLastError()) != hipSuccess) return hip_fail(he, "reduce launch");
    ph.mark(2, stream);

    int merge_grid = (int)((caps.heavy + kWavesPerBlock - 1) / kWavesPerBlock);
    if (merge_grid > device_cus(dev) * 8) merge_grid = device_cus(dev) * 8;
    if (merge_grid < 1) merge_grid = 1;
    hipLaunchKernelGGL((gt_reduce_merge_kernel<T, NVEC>), dim3(merge_grid), dim3(kBlock), 0, stream, rp);
    if ((he = hipGetLastError()) != hipSuccess) return hip_fail(he, "reduce merge launch");
    ph.commit(stream);
    return GT_SUCCESS;
}

using ReduceFn = gt_status (*)(const ReduceArgs&, const gt_tuning*, hipStream_t);

// Row sizes of 64 B .. 4 KiB: fp32 F in {16, ..., 1024}, bf16 F in {32, ..., 2048}.
template <typename T>
ReduceFn pick_reduce(int32_t F) {
    constexpr int EPV = 16 / Elt<T>::kBytes;
    if (F <= 0 || F % EPV != 0) return nullptr;
    switch (F / EPV) {
        case 4: return &launch_reduce<T, 4>;
        case 8: return &launch_reduce<T, 8>;
        case 16: return &launch_reduce<T, 16>;
        case 32: return &launch_reduce<T, 32>;
        case 64: return &launch_reduce<T, 64>;
        case 128: return &launch_reduce<T, 128>;
        case 256: return &launch_reduce<T, 256>;
        default: return nullptr;
    }
}
