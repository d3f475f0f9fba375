// Fused graph-transformer attention forward over a CSR graph, for gfx950.
//
// Operation: paper Section 2.2, attention family (iii) with graph-transformer
// logits; single streaming pass with online softmax (Section 3.2, Appendix
// D.2).  For every destination row i and head h:
//     out[i,h,:] = sum_e softmax_e(scale * <Q[i,h,:], K[j_e,h,:]>) V[j_e,h,:]
// The same skeleton evaluates the GATv2 layer of the same family (Section 2.2;
// Appendix D.2, fused GATv2 forward), selected by the KIND template argument:
//     out[i,h,:] = sum_e softmax_e(<a[h,:], LeakyReLU(L[i,h,:] + R[j_e,h,:])>) R[j_e,h,:]
// where each CSR entry gathers one row (R serves as key and value).
//
// Mapping (designed for 64-wide wavefronts, not taken from the paper's
// one-block-per-(node, head) CUDA layout):
//   * A node row of all heads, H*D elements, is R = H*D*sizeof(T) contiguous
//     bytes.  A lane group of G = min(64, R/16) lanes covers it with one
//     16-byte load per lane (NV = R/(16*G) loads when R > 1 KiB), so every
//     gathered K/V row is one fully coalesced request, and a wave holds
//     P = 64/G independent groups.
//   * A head's D elements occupy HL = D*sizeof(T)/16 consecutive lanes; the
//     score of a head is reduced across those lanes with DPP lane swaps.
//   * Degree-aware work split (Appendix B.1; Appendix D.1 for the chunked
//     heavy-node scheme): light rows get one group each, medium rows one wave
//     (the P groups split the row's entries and are merged across lanes),
//     heavy rows are cut into chunks processed by different waves whose
//     partial (max, sum, acc) states are merged in chunk order by a second
//     kernel, so results are bitwise reproducible and need no float atomics.
//   * Each group processes U entries per step: all U K-row and V-row loads
//     are issued before any is consumed, then one online-softmax update
//     covers the U entries (one rescale per step instead of one per entry).
//   * Neighbour indices are staged in LDS tiles loaded with one coalesced
//     4-byte load per lane.
//   * Light rows are assigned XCD-contiguously: the workgroups resident on
//     one XCD process one contiguous range of rows, so rows with shared
//     neighbourhoods (community-ordered ids) share that XCD's L2.

#include <hip/hip_runtime.h>

#include <array>
#include <atomic>
#include <climits>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <functional>
#include <map>
#include <type_traits>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "gt_attn.h"

// Workspace of the allocation-free entry point (gt_attn_fwd_noalloc): one
// array per device, held from the library's load until the process ends.
// Host code never passes `scratch` itself to a kernel (in host code the name
// is a stand-in, not a device address): it takes the device address from
// hipGetSymbolAddress once per device (scratch_of below).
constexpr size_t kScratchBytes = size_t(256) << 20;
static __device__ __align__(256) char scratch[kScratchBytes];

namespace {

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kBlock = kWave * kWavesPerBlock;
constexpr int kXcds = 8;

// Score kinds of the attention skeleton.
// KIND_GT_BF16W: the graph-transformer score with each softmax weight rounded
// to bf16 for P*V (bf16 rows pair two entries per dot2 instead of widening
// their value rows); an option for rows whose steps are arithmetic-bound.
enum { KIND_GT = 0, KIND_GATV2 = 1, KIND_GT_BF16W = 2 };

// Work-list counters in the workspace, cleared by a fill kernel at the start
// of each call.  Each counter sits on its own 256-byte line so that atomics
// on different counters do not serialise on one cache line.
//   CNT_MED, CNT_HEAVY, CNT_CHUNKS, CNT_SLOTS: medium rows, split rows, work
//     items, partial slots (list lengths, reserved with atomics);
//   CNT_OVERFLOW: set if a list capacity was exceeded (the CSR precondition
//     was violated; the excess entries are dropped);
//   CNT_LIGHT: nonzero if the light-row order holds any row (shapes that build
//     one); a flag written with plain stores;
//   CNT_WIN: byte 0 nonzero if some window was found dense, byte 1 if some
//     window was not (byte flags written with plain stores, read as one word).
enum {
    CNT_MED = 0, CNT_HEAVY = 1, CNT_CHUNKS = 2, CNT_OVERFLOW = 3, CNT_SLOTS = 4, CNT_LIGHT = 5, CNT_WIN = 6,
    CNT_COUNT = 7
};
constexpr int kCntStride = 64;                          // ints between counters
constexpr int kCntSetWords = CNT_COUNT * kCntStride;   // one counter set
#define CNT(c, i) ((c)[(i) * kCntStride])

struct bf16_tag {};

template <typename T> struct Elt;
template <> struct Elt<float> { static constexpr int kBytes = 4; };
template <> struct Elt<bf16_tag> { static constexpr int kBytes = 2; };

template <typename T, int H, int D>
struct Geo {
    static constexpr int kEB = Elt<T>::kBytes;
    static constexpr int kEPV = 16 / kEB;                   // elements per 16-B vector
    static constexpr int kRowBytes = H * D * kEB;           // one node row, all heads
    static constexpr int kNVec = kRowBytes / 16;
    static constexpr int kG = kNVec < kWave ? kNVec : kWave;  // lanes per group
    static constexpr int kNV = kNVec / kG;                  // 16-B vectors per lane
    static constexpr int kP = kWave / kG;                   // groups per wave
    static constexpr int kHL = D * kEB / 16;                // lanes per head (per vector slot)
    static constexpr int kU0 = (8 / kNV) > 2 ? (8 / kNV) : 2;
    static constexpr int kU = kU0 < kG ? kU0 : kG;          // entries per step per group
    static constexpr int kHD = H * D;
    static_assert(kRowBytes % 16 == 0, "row must be a whole number of 16-B vectors");
    static_assert(kHL >= 1 && kG % kHL == 0, "heads must tile the lane group");
    static_assert(kG % kU == 0 && kP * kU <= kWave, "index tiles must cover whole steps");
};

struct ChunkItem {
    int32_t row;
    int32_t slot;
    int64_t begin;
    int64_t end;
};

struct HeavyRow {
    int32_t row;
    int32_t base;  // first partial slot
    int32_t nch;   // number of chunks
    int32_t pad;
};

struct AttnParams {
    const int64_t* rowptr;
    const int32_t* colidx;
    const char* Q;
    const char* K;
    const char* V;
    char* out;
    float* lse;  // [N][H] natural-log logsumexp of the scaled scores, or nullptr
    int64_t N;
    float c;  // scale * log2(e); log2(e) for GATv2
    const float* att;  // GATv2 attention vector [H][D]
    float slope;       // GATv2 LeakyReLU negative slope
    int32_t light_max;
    int32_t cap_items;
    const int32_t* counters;
    const int32_t* med_list;
    const ChunkItem* chunks;
    float* part_acc;   // [slot][H*D]
    float2* part_ml;   // [slot][H]: (running max in log2 units, sum)
    const int32_t* light_list;  // [N]: light rows in step order per partition block, -1 elsewhere
};

struct PartParams {
    const int64_t* rowptr;
    int64_t N;
    int32_t light_max;
    int32_t heavy_min;
    int32_t chunk;
    int32_t cap_heavy;
    int32_t cap_items;  // work items: unsplit front rows + chunks of split rows
    int32_t cap_slots;  // partial-state slots: chunks of split rows only
    int32_t* counters;
    int32_t* med_list;
    HeavyRow* heavy;
    ChunkItem* chunks;
    int32_t* light_list = nullptr;  // or the block-local order of the light rows
    int32_t step = 1;               // entries per step of the light-row loop (its step classes)
    // Dense-tile windows (win_flags != nullptr): aligned 64-row windows whose
    // light rows are estimated to hold >= tile_min entries inside the window
    // are flagged for the tile kernel, and their light rows left out of the
    // light-row order.  The estimate reads one entry of every 8th light row.
    const int32_t* colidx = nullptr;
    uint8_t* win_flags = nullptr;  // [ceil(N / 64)]
    int32_t tile_min = 0;
    // the workspace's other counter set, zeroed by block 0 for the next call
    // that takes this workspace (nullptr: none)
    int32_t* zero_next = nullptr;
};

struct MergeParams {
    int32_t cap_heavy;
    const int32_t* counters;
    const HeavyRow* heavy;
    const float* part_acc;
    const float2* part_ml;
    char* out;
    float* lse;
};

// ------------------------------------------------------------ element codecs

template <typename T> __device__ __forceinline__ void widen(const uint4& r, float* f);

template <> __device__ __forceinline__ void widen<float>(const uint4& r, float* f) {
    f[0] = __uint_as_float(r.x);
    f[1] = __uint_as_float(r.y);
    f[2] = __uint_as_float(r.z);
    f[3] = __uint_as_float(r.w);
}

// bf16 element 2k sits in the low half of dword k (little endian); widening
// places the 16 bits in the upper half of an fp32 word, which is exact.
template <> __device__ __forceinline__ void widen<bf16_tag>(const uint4& r, float* f) {
    f[0] = __uint_as_float(r.x << 16);
    f[1] = __uint_as_float(r.x & 0xFFFF0000u);
    f[2] = __uint_as_float(r.y << 16);
    f[3] = __uint_as_float(r.y & 0xFFFF0000u);
    f[4] = __uint_as_float(r.z << 16);
    f[5] = __uint_as_float(r.z & 0xFFFF0000u);
    f[6] = __uint_as_float(r.w << 16);
    f[7] = __uint_as_float(r.w & 0xFFFF0000u);
}

// fp32 -> bf16 bits, round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint32_t bf16_rne(float x) {
    const uint32_t u = __float_as_uint(x);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

template <typename T> __device__ __forceinline__ uint4 narrow(const float* f);

template <> __device__ __forceinline__ uint4 narrow<float>(const float* f) {
    return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                      __float_as_uint(f[3]));
}

template <> __device__ __forceinline__ uint4 narrow<bf16_tag>(const float* f) {
    return make_uint4(bf16_rne(f[0]) | (bf16_rne(f[1]) << 16), bf16_rne(f[2]) | (bf16_rne(f[3]) << 16),
                      bf16_rne(f[4]) | (bf16_rne(f[5]) << 16), bf16_rne(f[6]) | (bf16_rne(f[7]) << 16));
}

// ---------------------------------------------------------- cross-lane sums

template <int CTRL> __device__ __forceinline__ float dpp(float x) {
    return __builtin_amdgcn_update_dpp(0.0f, x, CTRL, 0xF, 0xF, false);
}

// Sum over aligned groups of HL lanes; every lane of a group ends with the
// same bits (each step adds a pair of values in both orders, a+b == b+a).
template <int HL> __device__ __forceinline__ float head_sum(float x) {
    if constexpr (HL >= 2) x += dpp<0xB1>(x);    // quad_perm [1,0,3,2]: lane ^ 1
    if constexpr (HL >= 4) x += dpp<0x4E>(x);    // quad_perm [2,3,0,1]: lane ^ 2
    if constexpr (HL >= 8) x += dpp<0x141>(x);   // row_half_mirror: other quad of 8
    if constexpr (HL >= 16) x += dpp<0x140>(x);  // row_mirror: other half of 16
    if constexpr (HL >= 32) x += __shfl_xor(x, 16);
    if constexpr (HL >= 64) x += __shfl_xor(x, 32);
    return x;
}

// Sum of an int over the 64 lanes of a wavefront, in every lane (the head_sum
// pattern: DPP within rows of 16 lanes, then two cross-row swaps).
__device__ __forceinline__ int wave_sum_i32(int x) {
    x += __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false);   // lane ^ 1
    x += __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false);   // lane ^ 2
    x += __builtin_amdgcn_update_dpp(0, x, 0x141, 0xF, 0xF, false);  // other quad of 8
    x += __builtin_amdgcn_update_dpp(0, x, 0x140, 0xF, 0xF, false);  // other half of 16
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    return x;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Streaming 16-byte accesses for data touched once per call (the row vector,
// the output row): non-temporal, so they do not displace the gathered K/V rows
// that other rows reuse from L2 and the Infinity Cache.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_once(const char* p) {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return make_uint4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void store_once(char* p, const uint4& x) {
    const u32x4_t v = {x.x, x.y, x.z, x.w};
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4_t*>(p));
}

// bf16 pair arithmetic (gfx950 v_dot2c_f32_bf16, v_cvt_pk_bf16_f32, v_perm_b32).
// A dword holds bf16 element 2k in its low half and 2k+1 in its high half.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// c + a.lo * b.lo + a.hi * b.hi, products of bf16 pairs accumulated in fp32
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c,
                                           false);
}

// two fp32 values rounded to nearest even bf16, x in the low half
__device__ __forceinline__ uint32_t pack_bf16(float x, float y) {
    bf16x2_t r;
    r[0] = (__bf16)x;
    r[1] = (__bf16)y;
    return __builtin_bit_cast(uint32_t, r);
}

// (a.lo, b.lo) and (a.hi, b.hi): the same element of two rows as one pair
__device__ __forceinline__ uint32_t pair_lo(uint32_t a, uint32_t b) { return __builtin_amdgcn_perm(b, a, 0x05040100u); }
__device__ __forceinline__ uint32_t pair_hi(uint32_t a, uint32_t b) { return __builtin_amdgcn_perm(b, a, 0x07060302u); }

// Exponent-all-ones test of the eight bf16 values of v, folded into acc: a
// half's masked exponent plus 0x80 reaches bit 15 only when all eight exponent
// bits are set (Inf or NaN); the halves cannot carry into each other.  Any
// such value made bit 15 or 31 of acc set.
__device__ __forceinline__ uint32_t fold_nonfinite_bf16(uint32_t acc, const uint4& v) {
    acc |= (v.x & 0x7F807F80u) + 0x00800080u;
    acc |= (v.y & 0x7F807F80u) + 0x00800080u;
    acc |= (v.z & 0x7F807F80u) + 0x00800080u;
    acc |= (v.w & 0x7F807F80u) + 0x00800080u;
    return acc;
}

// Orders LDS traffic of one wavefront around a tile hand-off (the hardware
// executes a wave's LDS operations in order; this stops compiler reordering).
__device__ __forceinline__ void wave_lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

// ln(sum_e exp(s_e)) from the running state in base-2 units: the sum is
// 2^m * l, so the logarithm is (m + log2 l) * ln 2; -inf for an empty row.
__device__ __forceinline__ float lse_of(float m, float l) {
    return l > 0.0f ? (m + log2f(l)) * 0.6931471805599453f : -INFINITY;
}

// ------------------------------------------------------------ per-lane state

// One lane's share of a row's running state.  KIND_GT: q holds Q[i] and each
// entry loads K[j] (score) and V[j] (value).  KIND_GATV2: q holds L[i] and each
// entry loads only R[j], which gives both the score and the value.  The
// LeakyReLU term uses a * LeakyReLU(x) = a(1+s)/2 * x + a(1-s)/2 * |x| (exact
// for any slope s): a holds the lane's slice of a(1+s)/2 and a2 of a(1-s)/2,
// so an element costs one add and two FMAs (|x| is a free operand modifier)
// instead of a compare, a select and a multiply more.
// Entries per step of a row: the geometry's step, halved (8 -> 4) where short
// rows dominate the work of a step: for the GATv2 score, whose steps are
// arithmetic-heavy, and for rows narrow enough that a wave holds four or more
// of them.  A shorter step spends less on the padding of short rows and holds
// fewer registers.
template <typename T, int H, int D, int KIND>
struct StepOf {
    static constexpr int kU = Geo<T, H, D>::kU;
    static constexpr int value = ((KIND == KIND_GATV2 || Geo<T, H, D>::kP >= 4) && kU >= 8) ? kU / 2 : kU;
};

template <typename T, int H, int D, int KIND = KIND_GT>
struct RowState {
    using Gm = Geo<T, H, D>;
    static constexpr int kU = StepOf<T, H, D, KIND>::value;
    static constexpr bool kGat = KIND == KIND_GATV2;
    // bf16 graph-transformer rows: scores are bf16 dot2 on the raw Q and K
    // pairs, accumulated in fp32 (the products of bf16 pairs are exact).  P*V
    // widens the value rows exactly and multiplies them with the fp32 weights.
    // KIND_GT_BF16W pairs two entries instead: their weights are rounded to
    // one bf16 pair and a dot2 multiplies it with the same element of the two
    // entries' value rows (paired with v_perm), accumulating in fp32; that
    // halves the vector instructions of P*V, and each rounded weight is off by
    // at most the bf16 unit roundoff 2^-8, which bounds the extra error of out
    // by 2^-8 * sum_e p_e |v_e| / sum_e p_e.  Either way the normaliser (and
    // lse) sums the fp32 weights.  (GATv2 widens its gathered rows for the
    // score anyway.)
    static constexpr bool kDot2 = std::is_same<T, bf16_tag>::value && !kGat;
    static constexpr bool kPairPV = kDot2 && KIND == KIND_GT_BF16W;
    static_assert(!kPairPV || kU % 2 == 0, "dot2 pairs entries");
    float q[Gm::kNV][Gm::kEPV];
    float a[kGat ? Gm::kNV : 1][kGat ? Gm::kEPV : 1];
    float a2[kGat ? Gm::kNV : 1][kGat ? Gm::kEPV : 1];
    float acc[Gm::kNV][Gm::kEPV];
    float m[Gm::kNV];  // running max of log2-scaled scores for this lane's head
    float l[Gm::kNV];  // running sum of 2^(s - m)
    uint4 qraw[kDot2 ? Gm::kNV : 1];  // the row vector as bf16 pairs (dot2 form)

    __device__ __forceinline__ void begin(const char* __restrict__ Qb, int64_t row, int lig,
                                          const float* __restrict__ att = nullptr, float slope = 0.0f) {
        const char* qrow = Qb + row * (int64_t)Gm::kRowBytes + lig * 16;
#pragma unroll
        for (int k = 0; k < Gm::kNV; ++k) {
            const uint4 r = load_once(qrow + k * Gm::kG * 16);
            if constexpr (kDot2)
                qraw[k] = r;
            else
                widen<T>(r, q[k]);
            if constexpr (kGat) {
                // the attention vector is [H][D] fp32 in the row's element order
                const float* av = att + (lig + k * Gm::kG) * Gm::kEPV;
                const float hs = 0.5f * slope;
#pragma unroll
                for (int e = 0; e < Gm::kEPV; e += 4) {
                    const float4 x4 = *reinterpret_cast<const float4*>(av + e);
                    const float x[4] = {x4.x, x4.y, x4.z, x4.w};
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        a[k][e + t] = fmaf(hs, x[t], 0.5f * x[t]);
                        a2[k][e + t] = fmaf(-hs, x[t], 0.5f * x[t]);
                    }
                }
            }
            m[k] = -INFINITY;
            l[k] = 0.0f;
#pragma unroll
            for (int e = 0; e < Gm::kEPV; ++e) acc[k][e] = 0.0f;
        }
    }

    // begin() with this lane's 16-byte pieces of the row vector already in
    // registers (graph-transformer score only).
    __device__ __forceinline__ void begin_loaded(const uint4 (&r)[Gm::kNV]) {
        static_assert(!kGat, "the GATv2 state also needs its attention vector");
#pragma unroll
        for (int k = 0; k < Gm::kNV; ++k) {
            if constexpr (kDot2)
                qraw[k] = r[k];
            else
                widen<T>(r[k], q[k]);
            m[k] = -INFINITY;
            l[k] = 0.0f;
#pragma unroll
            for (int e = 0; e < Gm::kEPV; ++e) acc[k][e] = 0.0f;
        }
    }

    // Loads of one step: the K and V rows (GATv2: the R rows) of U entries,
    // 16 bytes per lane each.
    struct Batch {
        uint4 k[kU][Gm::kNV];
        uint4 v[kGat ? 1 : kU][Gm::kNV];
    };

    __device__ __forceinline__ void issue(const char* __restrict__ Kb, const char* __restrict__ Vb,
                                          const int32_t (&j)[kU], int lig, Batch& bt) const {
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int64_t off = (int64_t)j[u] * Gm::kRowBytes + lig * 16;
#pragma unroll
            for (int k = 0; k < Gm::kNV; ++k) {
                bt.k[u][k] = *reinterpret_cast<const uint4*>(Kb + off + k * Gm::kG * 16);
                if constexpr (!kGat) bt.v[u][k] = *reinterpret_cast<const uint4*>(Vb + off + k * Gm::kG * 16);
            }
        }
    }

    // Value row of entry u in vector slot k (GATv2: the gathered R row).
    __device__ __forceinline__ static const uint4& value(const Batch& bt, int u, int k) {
        if constexpr (kGat)
            return bt.k[u][k];
        else
            return bt.v[u][k];
    }

    // Score of entry u in vector slot k (log2 units, before masking).
    __device__ __forceinline__ float score(const Batch& bt, int u, int k, float c) const {
#pragma clang fp contract(off)
        float d = 0.0f;
        if constexpr (kDot2) {
            const uint4 kr = bt.k[u][k], qr = qraw[k];
            d = dot2_bf16(qr.x, kr.x, d);
            d = dot2_bf16(qr.y, kr.y, d);
            d = dot2_bf16(qr.z, kr.z, d);
            d = dot2_bf16(qr.w, kr.w, d);
        } else {
            float kf[Gm::kEPV];
            widen<T>(bt.k[u][k], kf);
            if constexpr (kGat) {
#pragma unroll
                for (int e = 0; e < Gm::kEPV; ++e) {
                    const float x = q[k][e] + kf[e];
                    d = fmaf(a[k][e], x, d);
                    d = fmaf(a2[k][e], fabsf(x), d);
                }
            } else {
#pragma unroll
                for (int e = 0; e < Gm::kEPV; ++e) d = fmaf(q[k][e], kf[e], d);
            }
        }
        return head_sum<Gm::kHL>(d) * c;
    }

    // Online-softmax update with the U entries of a batch; entries u >= nvalid
    // are copies of valid indices and contribute nothing (score -inf, weight 0).
    // The maximal entry gets weight exactly 1 (also in bf16), and an entry of
    // weight 0 adds exactly 0, so a single-entry row returns its value exactly;
    // dot2 steps with an odd number of valid entries pair the last one with a
    // weight-0 copy.
    __device__ __forceinline__ void consume(const Batch& bt, int nvalid, float c) {
        // No implicit contraction: fusing the score product into the later
        // subtraction of the running max would give the maximal entry a weight
        // of 2^(rounding error) instead of exactly 1.
#pragma clang fp contract(off)
        constexpr int U = kU;
        float s[U][Gm::kNV];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int k = 0; k < Gm::kNV; ++k) {
                const float d = score(bt, u, k, c);  // unconditional: the head sum is cross-lane
                s[u][k] = (u < nvalid) ? d : -INFINITY;
            }
#pragma unroll
        for (int k = 0; k < Gm::kNV; ++k) {
            float mb = m[k];
#pragma unroll
            for (int u = 0; u < U; ++u) mb = fmaxf(mb, s[u][k]);
            const float corr = fast_exp2(m[k] - mb);  // 0 on the first step (m = -inf)
            l[k] *= corr;
#pragma unroll
            for (int e = 0; e < Gm::kEPV; ++e) acc[k][e] *= corr;
            if constexpr (kPairPV) {
#pragma unroll
                for (int u = 0; u < U; u += 2) {
                    const float p0 = fast_exp2(s[u][k] - mb), p1 = fast_exp2(s[u + 1][k] - mb);
                    l[k] += p0;  // the normaliser (and so lse) from the fp32 weights
                    l[k] += p1;
                    const uint32_t pp = pack_bf16(p0, p1);
                    const uint4 v0 = value(bt, u, k), v1 = value(bt, u + 1, k);
                    const uint32_t a0[4] = {v0.x, v0.y, v0.z, v0.w}, a1[4] = {v1.x, v1.y, v1.z, v1.w};
#pragma unroll
                    for (int x = 0; x < 4; ++x) {
                        acc[k][2 * x] = dot2_bf16(pp, pair_lo(a0[x], a1[x]), acc[k][2 * x]);
                        acc[k][2 * x + 1] = dot2_bf16(pp, pair_hi(a0[x], a1[x]), acc[k][2 * x + 1]);
                    }
                }
            } else {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const float pu = fast_exp2(s[u][k] - mb);
                    l[k] += pu;
                    float vf[Gm::kEPV];
                    widen<T>(value(bt, u, k), vf);
#pragma unroll
                    for (int e = 0; e < Gm::kEPV; ++e) acc[k][e] = fmaf(pu, vf[e], acc[k][e]);
                }
            }
            m[k] = mb;
        }
    }

    __device__ __forceinline__ void step(const char* __restrict__ Kb, const char* __restrict__ Vb,
                                         const int32_t (&j)[kU], int nvalid, int lig, float c) {
        Batch bt;
        issue(Kb, Vb, j, lig, bt);
        consume(bt, nvalid, c);
    }

    // Merge the state held by the lane `off` positions away (same vector
    // slots in another group of the wave).
    __device__ __forceinline__ void merge_xor(int off) {
#pragma clang fp contract(off)
#pragma unroll
        for (int k = 0; k < Gm::kNV; ++k) {
            const float mo = __shfl_xor(m[k], off);
            const float lo = __shfl_xor(l[k], off);
            const float mn = fmaxf(m[k], mo);
            const float ca = (m[k] == mn) ? 1.0f : fast_exp2(m[k] - mn);
            const float cb = (mo == mn) ? 1.0f : fast_exp2(mo - mn);
            l[k] = l[k] * ca + lo * cb;
#pragma unroll
            for (int e = 0; e < Gm::kEPV; ++e) {
                const float ao = __shfl_xor(acc[k][e], off);
                acc[k][e] = acc[k][e] * ca + ao * cb;
            }
            m[k] = mn;
        }
    }

    __device__ __forceinline__ void store_out(char* __restrict__ outb, float* __restrict__ lse, int64_t row,
                                              int lig) const {
        char* orow = outb + row * (int64_t)Gm::kRowBytes + lig * 16;
#pragma unroll
        for (int k = 0; k < Gm::kNV; ++k) {
            const float inv = l[k] > 0.0f ? 1.0f / l[k] : 0.0f;
            float o[Gm::kEPV];
#pragma unroll
            for (int e = 0; e < Gm::kEPV; ++e) o[e] = acc[k][e] * inv;
            store_once(orow + k * Gm::kG * 16, narrow<T>(o));
            const int v = lig + k * Gm::kG;
            if (lse && v % Gm::kHL == 0) lse[row * H + v / Gm::kHL] = lse_of(m[k], l[k]);
        }
    }

    __device__ __forceinline__ void store_partial(float* __restrict__ pacc, float2* __restrict__ pml,
                                                  int32_t slot, int lig) const {
#pragma unroll
        for (int k = 0; k < Gm::kNV; ++k) {
            const int v = lig + k * Gm::kG;  // vector index within the row
            float* dst = pacc + (int64_t)slot * Gm::kHD + v * Gm::kEPV;
#pragma unroll
            for (int e = 0; e < Gm::kEPV; e += 4)
                *reinterpret_cast<float4*>(dst + e) =
                    make_float4(acc[k][e], acc[k][e + 1], acc[k][e + 2], acc[k][e + 3]);
            if (v % Gm::kHL == 0) pml[(int64_t)slot * H + v / Gm::kHL] = make_float2(m[k], l[k]);
        }
    }
};

// One wavefront streams CSR entries [b, e) of `row`; slot < 0 writes the
// normalised output, slot >= 0 writes the partial state of a chunk.
template <typename T, int H, int D, int KIND>
__device__ __forceinline__ void wave_segment(const AttnParams& p, int64_t row, int64_t b, int64_t e,
                                             int32_t slot, int32_t* __restrict__ tile, int lane) {
    using Gm = Geo<T, H, D>;
    constexpr int U = RowState<T, H, D, KIND>::kU, P = Gm::kP, G = Gm::kG;
    const int g = lane / G, lig = lane % G;
    RowState<T, H, D, KIND> st;
    st.begin(p.Q, row, lig, p.att, p.slope);
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
                st.step(p.K, p.V, j, nvalid, lig, p.c);
            }
        }
    }
#pragma unroll
    for (int off = G; off < kWave; off <<= 1) st.merge_xor(off);
    if (g == 0) {
        if (slot < 0)
            st.store_out(p.out, p.lse, row, lig);
        else
            st.store_partial(p.part_acc, p.part_ml, slot, lig);
    }
}

// Light rows (degree <= light_max), one lane group per row.  Each group walks
// its sequence of rows software-pipelined: the next row's rowptr entries are
// loaded before the current row's work starts, and its first index tile is
// loaded while the current row's first K/V batch is in flight, so a short row
// costs about one memory latency instead of three (rowptr -> colidx -> K/V).
// An index tile holds LightTile<G>::kR * G entries (kR loads per lane).
// Light rows in the partition's step order pay where a wave holds four or more
// rows (its groups then wait on their longest row), and for the GATv2 score,
// whose steps are arithmetic-heavy, already at two.  For the graph-transformer
// score with one or two rows per wave the extra index load and the longer
// partition cost more than the balance gains.
template <typename T, int H, int D, int KIND = KIND_GT>
struct SortedLight {
    static constexpr bool value = Geo<T, H, D>::kP >= 4 || (KIND == KIND_GATV2 && Geo<T, H, D>::kP >= 2);
};

template <int G> struct LightTile {
    static constexpr int kR = G >= 64 ? 1 : 2;
    static constexpr int kEntries = kR * G;
};

template <typename T, int H, int D, int KIND>
__device__ __forceinline__ void light_rows(const AttnParams& p, int64_t it, int64_t it_end,
                                           int64_t stride, int g, int lig,
                                           int32_t* __restrict__ gtile) {
    using Gm = Geo<T, H, D>;
    constexpr int U = RowState<T, H, D, KIND>::kU, G = Gm::kG, P = Gm::kP;
    constexpr int R = LightTile<G>::kR, TE = LightTile<G>::kEntries;
    static_assert(TE % U == 0, "index tiles hold whole steps");
    // entries [tb, tb + TE) of a row ending at ce (clamped to its last entry)
    auto load_tile = [&](int64_t tb, int64_t ce, int32_t (&v)[R]) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int64_t pos = tb + r * G + lig;
            v[r] = p.colidx[pos < ce ? pos : ce - 1];
        }
    };
    // Item `it` is the group's row at position it * P + g of the light-row
    // order (-1: none); the entry two items ahead is requested one item early,
    // so that it is in a register when its row pointers are needed.
    auto row_at = [&](int64_t i) -> int64_t {
        const int64_t pos = i * P + g;
        if constexpr (SortedLight<T, H, D, KIND>::value)
            return (i < it_end && pos < p.N) ? (int64_t)p.light_list[pos] : -1;
        else
            return (i < it_end && pos < p.N) ? pos : -1;
    };
    int64_t row = row_at(it);
    int64_t row_next = row_at(it + stride);
    bool ok = row >= 0;
    int64_t b = ok ? p.rowptr[row] : 0, e = ok ? p.rowptr[row + 1] : 0;
    bool mine = ok && (e - b) <= p.light_max;
    int32_t idx[R] = {};
    if (mine && e > b) load_tile(b, e, idx);
    while (it < it_end) {
        const int64_t crow = row, cb = b, ce = e;
        const bool cmine = mine;
        int32_t tv[R];
#pragma unroll
        for (int r = 0; r < R; ++r) tv[r] = idx[r];
        it += stride;
        row = row_next;
        row_next = row_at(it + stride);
        ok = row >= 0;
        b = ok ? p.rowptr[row] : 0;
        e = ok ? p.rowptr[row + 1] : 0;
        mine = ok && (e - b) <= p.light_max;
        bool fetched = false;
        if (cmine) {
            RowState<T, H, D, KIND> st;
            st.begin(p.Q, crow, lig, p.att, p.slope);
            for (int64_t tb = cb; tb < ce; tb += TE) {
                if (tb != cb) load_tile(tb, ce, tv);
                wave_lds_fence();
#pragma unroll
                for (int r = 0; r < R; ++r) gtile[r * G + lig] = tv[r];
                wave_lds_fence();
                const int nt = (int)((ce - tb) < TE ? (ce - tb) : TE);
                for (int t = 0; t < nt; t += U) {
                    const int nvalid = nt - t < U ? nt - t : U;
                    int32_t j[U];
#pragma unroll
                    for (int u = 0; u < U; ++u) j[u] = gtile[t + u];
                    typename RowState<T, H, D, KIND>::Batch bt;
                    st.issue(p.K, p.V, j, lig, bt);
                    if (!fetched) {  // next row's first tile, overlapped with this batch
                        if (mine && e > b) load_tile(b, e, idx);
                        fetched = true;
                    }
                    st.consume(bt, nvalid, p.c);
                }
            }
            st.store_out(p.out, p.lse, crow, lig);
        }
        if (!fetched && mine && e > b) load_tile(b, e, idx);
    }
}

// Attention kernel: first the chunk items (pieces of heavy rows,
// then whole medium rows), one wavefront each; then the light rows, P per
// wavefront, in XCD-contiguous ranges.
template <typename T, int H, int D, int KIND>
__global__ void __launch_bounds__(kBlock) gt_attn_kernel(AttnParams p) {
    using Gm = Geo<T, H, D>;
    // per wave: one 64-entry tile (wave items) or P light-row tiles
    constexpr int kTileWords = Gm::kP * LightTile<Gm::kG>::kEntries > kWave ? Gm::kP * LightTile<Gm::kG>::kEntries : kWave;
    __shared__ int32_t tiles[kWavesPerBlock][kTileWords];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x / kWave;
    int32_t* tile = tiles[wv];

    // Counts come from the partition kernel; clamping keeps every list read
    // inside the workspace even if the CSR precondition were violated.  The
    // light-row flag is read with them, so that a workgroup with nothing to
    // do ends after one round trip.
    const int32_t n_chunks = min(CNT(p.counters, CNT_CHUNKS), p.cap_items);
    const int32_t n_items = n_chunks + (int32_t)min((int64_t)CNT(p.counters, CNT_MED), p.N);
    const bool any_light = !SortedLight<T, H, D, KIND>::value || CNT(p.counters, CNT_LIGHT) != 0;
    const int nwaves = gridDim.x * kWavesPerBlock;
    for (int it = blockIdx.x * kWavesPerBlock + wv; it < n_items; it += nwaves) {
        if (it < n_chunks) {
            const ChunkItem ci = p.chunks[it];
            wave_segment<T, H, D, KIND>(p, ci.row, ci.begin, ci.end, ci.slot, tile, lane);
        } else {
            const int64_t row = p.med_list[it - n_chunks];
            wave_segment<T, H, D, KIND>(p, row, p.rowptr[row], p.rowptr[row + 1], -1, tile, lane);
        }
    }

    const int xcd = blockIdx.x % kXcds;
    const int waves_per_xcd = (gridDim.x / kXcds) * kWavesPerBlock;
    const int lw = (blockIdx.x / kXcds) * kWavesPerBlock + wv;
    const int64_t n_light = (p.N + Gm::kP - 1) / Gm::kP;
    const int64_t lo = n_light * xcd / kXcds, hi = n_light * (xcd + 1) / kXcds;
    const int g = lane / Gm::kG, lig = lane % Gm::kG;
    // (with a light-row order, it can be empty: every light row lies in a
    // dense window of the tile kernel)
    if (!any_light) return;
    light_rows<T, H, D, KIND>(p, lo + lw, hi, waves_per_xcd, g, lig, tile + g * LightTile<Gm::kG>::kEntries);
}

// ------------------------------------------------------- dense-tile path
//
// Locally dense windows (Section 3.3 and Appendix D.3 of the paper pack local
// neighbourhoods into tiles for matrix cores; this is a gfx950 design of the
// same idea, not the paper's 16x8 TCB format).  Rows are grouped in aligned
// windows of 64; the window's own 64 ids are its tile columns.  The partition
// kernel flags the windows whose light rows it estimates to be dense (a
// sample of one entry in every 8th light row); this kernel takes every light
// row of a flagged window (one workgroup per window), the CSR kernel every
// other row:
//   1. stage the window's rowptr, its K rows and its V rows (transposed) in
//      LDS with independent loads, and each light row's entries in registers;
//   2. per light row, a 64-bit mask of its in-window entries (a row with a
//      repeated in-window entry cannot be a mask and does not use the tile);
//   3. if the window holds at least `min_entries` masked entries and its V
//      tile only finite values, per head and per 16-row strip (one wave each):
//        S^T = K_w Q_strip^T  (bf16 MFMA 16x16x32, fp32 accumulate),
//      masked row-wise softmax statistics, and acc = P V_w (MFMA with P as
//      the sum of two bf16 terms, so the weights keep 16 significant bits;
//      with the bf16-weight option, one MFMA on P rounded to bf16); the
//      normaliser and lse sum the fp32 weights;
//   4. every light row then streams its remaining entries (all of them for a
//      row without a tile) with the CSR online-softmax step, continuing from
//      the tile's (m, l, acc), and writes its output.
// Non-light rows are left to the wave items of the CSR kernel.
//
// MFMA operand layout of v_mfma_f32_16x16x32_bf16 (64 lanes, l = lane):
//   A (16x32): lane l holds A[l%16][8*(l/16) + j], j = 0..7
//   B (32x16): lane l holds B[8*(l/16) + j][l%16]
//   C (16x16): lane l holds C[4*(l/16) + i][l%16], i = 0..3

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kWin = 64;          // window rows = tile columns
constexpr int kWinMaxDeg = 64;    // light rows handled here have at most this degree
constexpr int kNoTile = -(1 << 28);  // a wave's window count that rules the tile out
// Padded row of the transposed V tile, in bf16 elements: 34 dwords, so that
// the 16 rows one P*V operand load reads (8 bytes per lane) start 2 banks
// apart and cover all 32 banks once (a 36-dword row put rows n and n + 8 on
// the same banks).
constexpr int kVtStride = 68;

struct TileParams {
    const int64_t* rowptr;
    const int32_t* colidx;
    const char* Q;
    const char* K;
    const char* V;
    char* out;
    float* lse;
    int64_t N;
    float c;  // scale * log2(e)
    int32_t light_max;  // <= kWinMaxDeg
    int32_t min_entries;
    const uint8_t* win_flags;  // [ceil(N / 64)]: 1 for the dense windows the partition found
    const int32_t* counters;   // CNT_WIN: any window dense (byte 0) / not dense (byte 1)
};

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, m);
    const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), m);
    return ((uint64_t)hi << 32) | lo;
}

template <int H, int D>
struct TileLds {
    static constexpr int HD = H * D;
    static constexpr int KST = HD + 8;  // padded K row (bf16 elements)
    int64_t rp[kWin + 1];
    uint64_t masks[kWin];
    int32_t wave_cnt[kWavesPerBlock];
    // The K and V tiles are dead once the products are done; the strip results
    // and the index tiles of the remaining-entry stream then reuse their space.
    union alignas(16) {
        struct {
            uint16_t k[kWin][KST];
            uint16_t vt[HD][kVtStride];
        } kv;
        struct {
            float acc[kWavesPerBlock][16][HD + 4];  // padded: the MFMA-layout writes hit distinct banks
            int32_t ctile[kWavesPerBlock][kWave / (H * D / 8) * kWinMaxDeg];  // per lane group: one row's entries
        } rest;
    } big;
    float2 ml[kWavesPerBlock][16][H];
};

// Four workgroups per CU fit the LDS of a window (about 40 KB) when H*D <= 128
// and H <= 2; those shapes are held to 128 VGPRs so that registers allow it too.
// The stream stage of the tile kernel takes the row vectors of its rows from
// the strip's MFMA operand registers by cross-lane moves instead of reading Q
// a second time (on the SBM workload: 268 MB less fetched, about 10 us per
// call); for the 1x128 fp32-weight shape that holds 16 more registers across
// the products and spills, so it reads Q again.
template <int H, int D, int KIND>
struct QFromOperands {
    static constexpr bool value = !(H == 1 && D == 128 && KIND == KIND_GT);
};

template <int H, int D>
struct TileWaves {
    static constexpr int value = H <= 2 ? 4 : 1;
};

template <int H, int D, int KIND>
__global__ void __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(TileWaves<H, D>::value)))
gt_tile_kernel(TileParams p) {
    using Gm = Geo<bf16_tag, H, D>;
    using L = TileLds<H, D>;
    using RS = RowState<bf16_tag, H, D, KIND>;
    constexpr int HD = H * D;
    constexpr int G = Gm::kG, P = Gm::kP, U = RS::kU;
    // fp32 weights (KIND_GT): P = hi + lo as two bf16 terms, two P*V
    // products, |P - hi - lo| <= 2^-17 P; KIND_GT_BF16W: P rounded to bf16
    constexpr bool kSplitP = KIND == KIND_GT;
    static_assert(HD <= 128 && D % 32 == 0, "tile path shapes");
    __shared__ __attribute__((aligned(16))) L lds;

    const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
    const int g16 = lane >> 4, n16 = lane & 15;  // MFMA lane coordinates
    // Workgroup b takes window b if the partition flagged it dense and returns
    // at once otherwise.  The word of window flags (one word every workgroup
    // reads, so a cached one) is loaded first: with no dense window, the
    // workgroup ends there; with no sparse one, the window's own flag is not
    // needed; otherwise it is read after the row-bound loads are issued.  (A
    // persistent loop over a list of the dense windows measured slower: it
    // raised the kernel's register pressure past its 128-VGPR budget and
    // spilled; a list also needs its entry before any other load.)
    const int64_t r0 = (int64_t)blockIdx.x * kWin;
    const int64_t wend = r0 + kWin;
    const int32_t win_state = CNT(p.counters, CNT_WIN);
    if ((win_state & 0xFF) == 0) return;
    const bool all_dense = (win_state & 0xFF00) == 0;

    // bounds of this lane's row in the mask stage (4 lanes per row), loaded
    // first so that its entries can be requested right after the staging loads
    const int srow = lane >> 2, sub = lane & 3;
    const int wrow = 16 * wv + srow;  // row within the window
    const int64_t r = r0 + wrow;
    // (rows past the end read rowptr[N] twice: an empty row.  The loads of
    // this stage are unconditional, with clamped addresses, so that the
    // compiler can wait for the row bounds alone while the later staging loads
    // are still in flight.)
    const int64_t mb = p.rowptr[r < p.N ? r : p.N];
    const int64_t me = p.rowptr[r + 1 < p.N ? r + 1 : p.N];
    if (!all_dense && !p.win_flags[blockIdx.x]) return;

    // ---- 1. staging.  Every load of the stage is issued before any LDS write,
    // with compile-time trip counts: the window's rowptr entries, its K and V
    // pieces and this lane's strip row of Q go out together, then the entries
    // of the mask stage (which wait only for the row bounds above), and only
    // then do the LDS writes wait for their data.  So staging a window costs
    // about two memory latencies (row bounds, then entries), not one per loop
    // trip.
    constexpr int kKPieces = kWin * (HD / 8);        // 16-byte pieces of the K tile
    constexpr int kVPieces = (kWin / 2) * (HD / 8);  // pieces of the row pairs of the V tile
    constexpr int kKIt = (kKPieces + kBlock - 1) / kBlock;
    constexpr int kVIt = (kVPieces + kBlock - 1) / kBlock;
    static_assert(kKPieces % kBlock == 0, "the K tile is a whole number of workgroup loads");
    // Rows past the end read the last row instead: their K columns and Q rows
    // are masked out of every score, and their V columns are zeroed when the
    // tile is written (a weight of 0 must not meet a non-finite value).  No
    // loaded register is overwritten before it arrives, which would make the
    // load wait at once.
    const int64_t last = p.N - 1;
    const int64_t rpv = p.rowptr[(r0 + tid < p.N) ? r0 + tid : p.N];
    uint4 kx[kKIt];
#pragma unroll
    for (int it = 0; it < kKIt; ++it) {
        // K rows as they are: 16 bytes of one row per lane
        const int v = tid + it * kBlock, cc = v % kWin, e0 = (v / kWin) * 8;
        const int64_t rk = r0 + cc;
        kx[it] = *reinterpret_cast<const uint4*>(p.K + ((rk < p.N ? rk : last) * HD + e0) * 2);
    }
    uint4 va[kVIt], vb[kVIt];
#pragma unroll
    for (int it = 0; it < kVIt; ++it) {
        // V transposed: a lane takes 8 elements of two consecutive rows (the
        // 1x32 shape has fewer pieces than lanes: the rest load piece 0)
        const int v0 = tid + it * kBlock;
        const int v = (kVPieces % kBlock == 0 || v0 < kVPieces) ? v0 : 0;
        const int pc = v % (kWin / 2), e0 = (v / (kWin / 2)) * 8;
        const int64_t ra = r0 + 2 * pc;
        va[it] = *reinterpret_cast<const uint4*>(p.V + ((ra < p.N ? ra : last) * HD + e0) * 2);
        vb[it] = *reinterpret_cast<const uint4*>(p.V + ((ra + 1 < p.N ? ra + 1 : last) * HD + e0) * 2);
    }
    // this lane's strip row of Q (all heads), as MFMA B operands
    const int64_t qrow = r0 + 16 * wv + n16;
    uint4 qreg[HD / 32];
#pragma unroll
    for (int t = 0; t < HD / 32; ++t) {
        qreg[t] = *reinterpret_cast<const uint4*>(p.Q + ((qrow < p.N ? qrow : last) * HD + 32 * t + 8 * g16) * 2);
    }

    // ---- 2. in-window masks: 4 lanes per row, 16 rows per wave.  The entries
    // come straight from colidx (one batch of independent loads, behind the
    // staging loads); the remaining-entry stream reads them again later, so
    // the window needs no LDS copy of its entries.
    const bool light = r < p.N && (me - mb) <= p.light_max;
    constexpr int kMaskPer = kWinMaxDeg / 4;  // entries per lane (light_max <= kWinMaxDeg)
    int32_t ent[kMaskPer] = {};
    if (light && me > mb) {
#pragma unroll
        for (int k = 0; k < kMaskPer; ++k) {
            const int64_t pos = mb + sub + 4 * k;
            ent[k] = p.colidx[pos < me ? pos : me - 1];
        }
    }
    // the staged tiles to LDS (read after the barrier below)
    if (tid <= kWin) lds.rp[tid] = rpv;
#pragma unroll
    for (int it = 0; it < kKIt; ++it) {
        const int v = tid + it * kBlock, cc = v % kWin, e0 = (v / kWin) * 8;
        *reinterpret_cast<uint4*>(&lds.big.kv.k[cc][e0]) = r0 + cc < p.N ? kx[it] : make_uint4(0, 0, 0, 0);
    }
    // Inf or NaN anywhere in the value tile: P*V sums over every column of
    // the window, and a weight of 0 times such a value is NaN, so one row's
    // value would leak into rows that do not reference it.  Such a window is
    // streamed instead (below).
    uint32_t vbits = 0;
#pragma unroll
    for (int it = 0; it < kVIt; ++it) {
        // each element pair as one dword, so the 32 lanes of a row pair write 32
        // consecutive dwords of one vt row
        const int v = tid + it * kBlock, pc = v % (kWin / 2), e0 = (v / (kWin / 2)) * 8;
        if (kVPieces % kBlock == 0 || v < kVPieces) {
            const int64_t ra = r0 + 2 * pc;
            const uint4 a = ra < p.N ? va[it] : make_uint4(0, 0, 0, 0);
            const uint4 b = ra + 1 < p.N ? vb[it] : make_uint4(0, 0, 0, 0);
            vbits = fold_nonfinite_bf16(fold_nonfinite_bf16(vbits, a), b);
            const uint32_t wa[4] = {a.x, a.y, a.z, a.w}, wb[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                *reinterpret_cast<uint32_t*>(&lds.big.kv.vt[e0 + 2 * q][2 * pc]) = pair_lo(wa[q], wb[q]);
                *reinterpret_cast<uint32_t*>(&lds.big.kv.vt[e0 + 2 * q + 1][2 * pc]) = pair_hi(wa[q], wb[q]);
            }
        }
    }
    uint64_t mk = 0;
    int cnt = 0;
    if (light) {
#pragma unroll
        for (int k = 0; k < kMaskPer; ++k) {
            const int64_t j = ent[k];
            if (mb + sub + 4 * k < me && j >= r0 && j < wend) {
                mk |= 1ull << (j - r0);
                ++cnt;
            }
        }
    }
    mk |= shfl_xor_u64(mk, 1);
    mk |= shfl_xor_u64(mk, 2);
    cnt += __shfl_xor(cnt, 1);
    cnt += __shfl_xor(cnt, 2);
    const bool tile_ok = light && __popcll(mk) == cnt;  // no repeated in-window entry
    if (sub == 0) lds.masks[wrow] = tile_ok ? mk : 0;
    int wc = (sub == 0 && tile_ok) ? cnt : 0;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) wc += __shfl_xor(wc, o);
    // a wave that staged a non-finite value puts the window's count far below
    // any threshold
    const bool v_nonfinite = __ballot((vbits & 0x80008000u) != 0) != 0;
    if (lane == 0) lds.wave_cnt[wv] = v_nonfinite ? kNoTile : wc;
    const uint64_t ok_bits = __ballot(sub == 0 && tile_ok);     // bit 4*sr: strip row sr
    const uint64_t light_bits = __ballot(sub == 0 && light);
    __syncthreads();
    int total = 0;
#pragma unroll
    for (int w = 0; w < kWavesPerBlock; ++w) total += lds.wave_cnt[w];
    const bool dense = total >= p.min_entries;  // uniform over the workgroup

    // ---- 3. tiles
    float mx[H], lsum[H];
    f32x4_t oacc[H][D / 16];
    if (dense) {
        const uint64_t rmask = lds.masks[16 * wv + n16];
#pragma unroll
        for (int h = 0; h < H; ++h) {
            f32x4_t sacc[4];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) sacc[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < D / 32; ++ks) {
                const bf16x8_t bq = __builtin_bit_cast(bf16x8_t, qreg[(h * D) / 32 + ks]);
#pragma unroll
                for (int mt = 0; mt < 4; ++mt) {
                    const bf16x8_t ak = __builtin_bit_cast(
                        bf16x8_t, *reinterpret_cast<const uint4*>(&lds.big.kv.k[16 * mt + n16][h * D + 32 * ks + 8 * g16]));
                    sacc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ak, bq, sacc[mt], 0, 0, 0);
                }
            }
            // lane holds S[strip row n16][window column 16*mt + 4*g16 + i] = sacc[mt][i]
            float pr[16];
            float m = -INFINITY;
            {
#pragma clang fp contract(off)
#pragma unroll
                for (int mt = 0; mt < 4; ++mt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int cc = 16 * mt + 4 * g16 + i;
                        const float sv = ((rmask >> cc) & 1ull) ? sacc[mt][i] * p.c : -INFINITY;
                        pr[4 * mt + i] = sv;
                        m = fmaxf(m, sv);
                    }
                m = fmaxf(m, __shfl_xor(m, 16));
                m = fmaxf(m, __shfl_xor(m, 32));
            }
            uint32_t pb[16], pl[kSplitP ? 16 : 1];
            float ls = 0.0f;
#pragma unroll
            for (int t = 0; t < 16; ++t) {
                const float pv = (m == -INFINITY) ? 0.0f : fast_exp2(pr[t] - m);
                pb[t] = bf16_rne(pv);
                // pv - hi is exact in fp32; its bf16 rounding is the low term
                if constexpr (kSplitP) pl[t] = bf16_rne(pv - __uint_as_float(pb[t] << 16));
                ls += pv;  // the normaliser (and lse) from the fp32 weights
            }
            ls += __shfl_xor(ls, 16);
            ls += __shfl_xor(ls, 32);
            mx[h] = m;
            lsum[h] = ls;
            // acc = P V_w; K order of step ks, slot 8*g16 + j: window column
            // 16*(2ks + j/4) + 4*g16 + j%4, i.e. exactly the weights this lane holds
#pragma unroll
            for (int dt = 0; dt < D / 16; ++dt) oacc[h][dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const uint4 au = make_uint4(pb[8 * ks + 0] | (pb[8 * ks + 1] << 16), pb[8 * ks + 2] | (pb[8 * ks + 3] << 16),
                                            pb[8 * ks + 4] | (pb[8 * ks + 5] << 16), pb[8 * ks + 6] | (pb[8 * ks + 7] << 16));
                const bf16x8_t ap = __builtin_bit_cast(bf16x8_t, au);
                bf16x8_t apl = ap;
                if constexpr (kSplitP)
                    apl = __builtin_bit_cast(
                        bf16x8_t, make_uint4(pl[8 * ks + 0] | (pl[8 * ks + 1] << 16), pl[8 * ks + 2] | (pl[8 * ks + 3] << 16),
                                             pl[8 * ks + 4] | (pl[8 * ks + 5] << 16), pl[8 * ks + 6] | (pl[8 * ks + 7] << 16)));
#pragma unroll
                for (int dt = 0; dt < D / 16; ++dt) {
                    const int e = h * D + 16 * dt + n16;
                    const uint2 lo = *reinterpret_cast<const uint2*>(&lds.big.kv.vt[e][32 * ks + 4 * g16]);
                    const uint2 hi = *reinterpret_cast<const uint2*>(&lds.big.kv.vt[e][32 * ks + 16 + 4 * g16]);
                    const bf16x8_t bv = __builtin_bit_cast(bf16x8_t, make_uint4(lo.x, lo.y, hi.x, hi.y));
                    oacc[h][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap, bv, oacc[h][dt], 0, 0, 0);
                    if constexpr (kSplitP)
                        oacc[h][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(apl, bv, oacc[h][dt], 0, 0, 0);
                }
            }
        }
    }
    __syncthreads();  // K / V tiles no longer read: their LDS now holds the strip results
    if (dense) {
#pragma unroll
        for (int h = 0; h < H; ++h) {
#pragma unroll
            for (int dt = 0; dt < D / 16; ++dt)
#pragma unroll
                for (int i = 0; i < 4; ++i) lds.big.rest.acc[wv][4 * g16 + i][h * D + 16 * dt + n16] = oacc[h][dt][i];
            if (g16 == 0) lds.ml[wv][n16][h] = make_float2(mx[h], lsum[h]);
        }
    }
    wave_lds_fence();

    // ---- 4. remaining entries of each light row, CSR online softmax, output.
    // Each lane group takes rows g, g + P, ... of the wave's strip; the entries
    // of a group's next row are requested before the current row's gathers.
    const int g = lane / G, lig = lane % G;
    int32_t* gtile = lds.big.rest.ctile[wv] + g * kWinMaxDeg;
    constexpr int kRowPer = (kWinMaxDeg + G - 1) / G;  // a light row: at most kWinMaxDeg entries
    constexpr int kPasses = 16 / P;
    // The row vector of the group's row of a pass, from the strip's MFMA
    // operands (lane 16*g16 + n16 of qreg[t] holds elements 32t + 8*g16 .. + 7
    // of strip row n16) by cross-lane moves, rather than a second read from
    // memory.  Taken at the top of each pass, where every lane is active (a
    // move reads zero from an inactive lane), with selects rather than
    // branches.
    constexpr bool kQRegs = QFromOperands<H, D, KIND>::value;
    auto row_vector = [&](int pass, uint4 (&qp)[Gm::kNV]) {
#pragma unroll
        for (int k = 0; k < Gm::kNV; ++k) {
            const int e0 = 8 * (lig + k * G);  // first element of this lane's piece
            const int src = 16 * ((e0 % 32) / 8) + pass * P + g, tsel = e0 / 32;
            uint32_t v[4] = {0, 0, 0, 0};
#pragma unroll
            for (int t = 0; t < HD / 32; ++t) {
                const uint32_t x[4] = {(uint32_t)__shfl((int)qreg[t].x, src), (uint32_t)__shfl((int)qreg[t].y, src),
                                       (uint32_t)__shfl((int)qreg[t].z, src), (uint32_t)__shfl((int)qreg[t].w, src)};
#pragma unroll
                for (int c = 0; c < 4; ++c) v[c] = tsel == t ? x[c] : v[c];
            }
            qp[k] = make_uint4(v[0], v[1], v[2], v[3]);
        }
    };
    auto load_entries = [&](int pass, int32_t (&e)[kRowPer]) {
        const int sr = pass * P + g, wr = 16 * wv + sr;
        const int64_t eb = lds.rp[wr], ee = lds.rp[wr + 1];
        if (((light_bits >> (4 * sr)) & 1ull) && ee > eb) {
#pragma unroll
            for (int k = 0; k < kRowPer; ++k) {
                const int64_t pos = eb + lig + k * G;
                e[k] = p.colidx[pos < ee ? pos : ee - 1];
            }
        }
    };
    int32_t nxt[kRowPer] = {};
    load_entries(0, nxt);
    for (int pass = 0; pass < kPasses; ++pass) {
        int32_t re[kRowPer];
#pragma unroll
        for (int k = 0; k < kRowPer; ++k) re[k] = nxt[k];
        if (pass + 1 < kPasses) load_entries(pass + 1, nxt);
        uint4 qp[Gm::kNV];
        if constexpr (kQRegs) row_vector(pass, qp);
        const int sr = pass * P + g;
        if (!((light_bits >> (4 * sr)) & 1ull)) continue;
        const bool use_tile = dense && ((ok_bits >> (4 * sr)) & 1ull);
        const int wr = 16 * wv + sr;
        const int64_t row = r0 + wr;
        RS st;
        if constexpr (kQRegs)
            st.begin_loaded(qp);
        else
            st.begin(p.Q, row, lig);
        if (use_tile) {
#pragma unroll
            for (int k = 0; k < Gm::kNV; ++k) {
                const int v = lig + k * G;
                const float2 ml = lds.ml[wv][sr][v / Gm::kHL];
                st.m[k] = ml.x;
                st.l[k] = ml.y;
#pragma unroll
                for (int q = 0; q < Gm::kEPV; ++q) st.acc[k][q] = lds.big.rest.acc[wv][sr][v * Gm::kEPV + q];
            }
        }
        // the row's remaining entries (outside the tile) into gtile
        const int64_t eb = lds.rp[wr], ee = lds.rp[wr + 1];
        int n_take = 0;
#pragma unroll
        for (int k = 0; k < kRowPer; ++k) {
            const bool in = eb + lig + k * G < ee;
            const int32_t idx = re[k];
            const bool take = in && !(use_tile && idx >= r0 && idx < wend);
            const uint64_t bal = __ballot(take);
            const uint32_t gbits = (uint32_t)((bal >> (g * G)) & ((1ull << G) - 1));
            if (take) gtile[n_take + __popc(gbits & ((1u << lig) - 1u))] = idx;
            n_take += __popc(gbits);
        }
        wave_lds_fence();
        for (int t = 0; t < n_take; t += U) {
            const int nvalid = n_take - t < U ? n_take - t : U;
            int32_t j[U];
#pragma unroll
            for (int u = 0; u < U; ++u) j[u] = gtile[(t + u < n_take) ? t + u : n_take - 1];
            st.step(p.K, p.V, j, nvalid, lig, p.c);
        }
        wave_lds_fence();
        st.store_out(p.out, p.lse, row, lig);
    }
}

// Degree binning.  A block owns RPT * 256 contiguous rows; thread t takes
// rows t, t+256, ... of the block, so every rowptr load is coalesced.  Medium
// rows are compacted with wave ballots; heavy-row and chunk counts with block
// scans; each block then reserves its output ranges with one atomic per list.
// A heavy row is cut into at most kMaxChunks chunks of (about) equal length,
// at least `chunk` entries each, so the ordered merge of a hub stays a few
// load rounds long.
constexpr int kMaxChunks = 32;
constexpr int kLightClasses = 16;  // step-count classes of the light-row order

// Exclusive scans over the block of three per-thread counts at once (one
// barrier); totals in tot[0..2].
__device__ __forceinline__ int3 block_exclusive_scan3(int3 v, int3* lds_waves, int* tot) {
    const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
    int3 x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int a = __shfl_up(x.x, o), b = __shfl_up(x.y, o), c = __shfl_up(x.z, o);
        if (lane >= o) {
            x.x += a;
            x.y += b;
            x.z += c;
        }
    }
    if (lane == kWave - 1) lds_waves[wv] = x;
    __syncthreads();
    int3 before = make_int3(0, 0, 0);
    tot[0] = tot[1] = tot[2] = 0;
#pragma unroll
    for (int w = 0; w < kWavesPerBlock; ++w) {
        const int3 t = lds_waves[w];
        if (w < wv) {
            before.x += t.x;
            before.y += t.y;
            before.z += t.z;
        }
        tot[0] += t.x;
        tot[1] += t.y;
        tot[2] += t.z;
    }
    return make_int3(before.x + x.x - v.x, before.y + x.y - v.y, before.z + x.z - v.z);
}

__device__ __forceinline__ int chunks_of(int64_t deg, int chunk) {
    const int64_t n = (deg + chunk - 1) / chunk;
    return (int)(n < kMaxChunks ? n : kMaxChunks);
}

template <int RPT>
__global__ void __launch_bounds__(kBlock) gt_partition_kernel(PartParams p) {
    constexpr int kPartRowsPerThread = RPT;
    constexpr int kPartRowsPerBlock = kBlock * RPT;
    __shared__ int wave_cnt[kPartRowsPerThread][kWavesPerBlock];
    __shared__ int3 scan3[kWavesPerBlock];
    __shared__ int base[4];
    __shared__ int cls_cnt[kLightClasses], cls_pos[kLightClasses];
    __shared__ int win_dense[kPartRowsPerThread][kWavesPerBlock];  // dense-tile window flags of this block
    const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x / kWave;
    const int64_t r0 = (int64_t)blockIdx.x * kPartRowsPerBlock;
    int64_t rb[kPartRowsPerThread], deg[kPartRowsPerThread];
    bool med[kPartRowsPerThread];
    uint64_t mask[kPartRowsPerThread];
    int n_heavy = 0, n_chunk = 0, n_slot = 0;
    if (p.zero_next && blockIdx.x == 0)
        for (int i = threadIdx.x; i < kCntSetWords; i += kBlock) p.zero_next[i] = 0;
    if (p.light_list && threadIdx.x < kLightClasses) cls_cnt[threadIdx.x] = 0;
#pragma unroll
    for (int k = 0; k < kPartRowsPerThread; ++k) {
        const int64_t r = r0 + k * kBlock + threadIdx.x;
        rb[k] = 0;
        deg[k] = 0;
        if (r < p.N) {
            rb[k] = p.rowptr[r];
            deg[k] = p.rowptr[r + 1] - rb[k];
        }
        med[k] = deg[k] > p.light_max && deg[k] < p.heavy_min;
        mask[k] = __ballot(med[k]);
        if (lane == 0) wave_cnt[k][wv] = __popcll(mask[k]);
        if (deg[k] >= p.heavy_min) {
            const int nch = chunks_of(deg[k], p.chunk);
            n_heavy += nch > 1 ? 1 : 0;
            n_chunk += nch;
            n_slot += nch > 1 ? nch : 0;
        }
    }
    // Dense-tile windows.  In iteration k, wave wv holds the 64 rows of one
    // aligned window (r0 is a multiple of 1024).  The window's light rows hold
    // ld entries; every 8th light row contributes its middle entry as a
    // sample, and the in-window share of the sampled rows' entries (self-loops
    // not counted) estimates the window's in-window entries (the tile kernel
    // counts them exactly and still streams a window that falls short).  A dense window's light rows
    // belong to the tile kernel (tiled), all others stay on this path.
    bool tiled[kPartRowsPerThread];
#pragma unroll
    for (int k = 0; k < kPartRowsPerThread; ++k) tiled[k] = false;
    if (p.win_flags) {
        int32_t smp[kPartRowsPerThread];
#pragma unroll
        for (int k = 0; k < kPartRowsPerThread; ++k) {
            const int64_t r = r0 + k * kBlock + threadIdx.x;
            smp[k] = -1;
            if (r < p.N && deg[k] > 0 && deg[k] <= p.light_max && (lane & 7) == 0)
                smp[k] = p.colidx[rb[k] + deg[k] / 2];
        }
#pragma unroll
        for (int k = 0; k < kPartRowsPerThread; ++k) {
            const int64_t r = r0 + k * kBlock + threadIdx.x;
            const bool lt = r < p.N && deg[k] <= p.light_max;
            // light degrees are <= 64, so a window's sums fit: ld <= 4096 and
            // the sampled sums (8 rows) <= 512, packed two to a word
            const int ld = wave_sum_i32(lt ? (int)deg[k] : 0);
            // a sampled self-loop does not count: every row has at most one,
            // and rows holding only their self-loop would make sparse windows
            // look dense
            const int sd = smp[k] >= 0 ? (int)deg[k] : 0;
            const int si = (smp[k] >= 0 && smp[k] != r && ((int64_t)smp[k] >> 6) == (r >> 6)) ? sd : 0;
            const int ss = wave_sum_i32(sd | (si << 16));
            const int sd_w = ss & 0xFFFF, si_w = ss >> 16;
            const bool dense = p.tile_min <= 1 ? ld > 0
                                               : (ld >= p.tile_min && si_w > 0 &&
                                                  (int64_t)si_w * ld >= (int64_t)p.tile_min * sd_w);
            tiled[k] = dense && lt;
            const int64_t win = (r0 + k * kBlock + wv * kWave) >> 6;
            if (lane == 0) {
                const bool exists = win * kWave < p.N;
                if (exists) p.win_flags[win] = dense ? 1 : 0;
                win_dense[k][wv] = !exists ? 2 : dense ? 1 : 0;  // 2: past the last row
            }
        }
    }
    if (p.light_list) {
        // Light rows of this block in descending step count (a counting sort in
        // LDS), so the lane groups of a wave take rows of similar length and a
        // wave does not wait on one long row among short ones: the degree
        // bucketing of the degree-aware mapping (Appendix B.1), applied to the
        // rows that share a wavefront.  The order within
        // a step class is arbitrary; every row is computed on its own, so the
        // results do not depend on it.  Positions after the block's light rows
        // hold -1.
        __syncthreads();  // cls_cnt zeroed
        int cls[kPartRowsPerThread];
#pragma unroll
        for (int k = 0; k < kPartRowsPerThread; ++k) {
            const int64_t r = r0 + k * kBlock + threadIdx.x;
            cls[k] = -1;
            if (r < p.N && deg[k] <= p.light_max && !tiled[k]) {
                const int64_t st = (deg[k] + p.step - 1) / p.step;
                cls[k] = (int)(st < kLightClasses - 1 ? st : kLightClasses - 1);
                atomicAdd(&cls_cnt[cls[k]], 1);
            }
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            int acc = 0;
            for (int c = kLightClasses - 1; c >= 0; --c) {
                cls_pos[c] = acc;
                acc += cls_cnt[c];
            }
            cls_cnt[0] = acc;  // the block's light-row count (class 0's count is no longer needed)
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < kPartRowsPerThread; ++k)
            if (cls[k] >= 0) {
                const int at = atomicAdd(&cls_pos[cls[k]], 1);
                p.light_list[r0 + at] = (int32_t)(r0 + k * kBlock + threadIdx.x);
            }
        const int n_light_rows = cls_cnt[0];
        const int64_t rows_here = (p.N - r0 < kPartRowsPerBlock) ? p.N - r0 : kPartRowsPerBlock;
        for (int64_t j = n_light_rows + threadIdx.x; j < rows_here; j += kBlock) p.light_list[r0 + j] = -1;
    }
    int tots[3];
    const int3 offs = block_exclusive_scan3(make_int3(n_heavy, n_chunk, n_slot), scan3, tots);
    const int off_h = offs.x, off_c = offs.y, off_s = offs.z;
    // The block's reservations: lanes 0..3 of wave 0 each add to one list
    // counter, so the atomics go out together rather than one after another;
    // lanes 4..6 raise flags with plain stores.
    if (threadIdx.x < 7) {
        const int t = threadIdx.x;
        if (t < 4) {
            int amount = 0, which = CNT_MED;
            if (t == 0) {
                for (int k = 0; k < kPartRowsPerThread; ++k)
                    for (int w = 0; w < kWavesPerBlock; ++w) amount += wave_cnt[k][w];
            } else {
                amount = tots[t - 1];
                which = t == 1 ? CNT_HEAVY : t == 2 ? CNT_CHUNKS : CNT_SLOTS;
            }
            base[t] = amount ? atomicAdd(&CNT(p.counters, which), amount) : 0;
        } else if (t == 4) {
            // light rows left in the order: none lets the attention kernel
            // skip its light-row loop (every light row in dense windows)
            if (p.light_list && cls_cnt[0] > 0) CNT(p.counters, CNT_LIGHT) = 1;
        } else if (p.win_flags) {
            const int want = t == 5 ? 1 : 0;  // lane 5: a dense window; lane 6: a sparse one
            bool seen = false;
            for (int k = 0; k < kPartRowsPerThread; ++k)
                for (int w = 0; w < kWavesPerBlock; ++w) seen |= win_dense[k][w] == want;
            if (seen) reinterpret_cast<uint8_t*>(&CNT(p.counters, CNT_WIN))[t - 5] = 1;
        }
    }
    __syncthreads();
    int pos = base[0];
    int hid = base[1] + off_h, item = base[2] + off_c, slot = base[3] + off_s;
#pragma unroll
    for (int k = 0; k < kPartRowsPerThread; ++k) {
        const int64_t r = r0 + k * kBlock + threadIdx.x;
        int before = 0;
        for (int w = 0; w < wv; ++w) before += wave_cnt[k][w];
        if (med[k]) p.med_list[pos + before + __popcll(mask[k] & ((1ull << lane) - 1))] = (int32_t)r;
        for (int w = 0; w < kWavesPerBlock; ++w) pos += wave_cnt[k][w];
        if (deg[k] >= p.heavy_min) {
            // Rows of degree >= heavy_min are placed first in the work list (the
            // longest items start first).  A row that fits in one chunk is a
            // single item writing its output directly; a longer row is split,
            // its chunks get partial-state slots, and it is recorded for the
            // ordered merge.  Only split rows take slots, so the slots number
            // at most 2E/chunk (a split row of degree d > chunk has fewer than
            // 2d/chunk chunks).
            const int nch = chunks_of(deg[k], p.chunk);
            const int split = nch > 1 ? 1 : 0;
            if (hid + split > p.cap_heavy || item + nch > p.cap_items || (split && slot + nch > p.cap_slots)) {
                atomicOr(&CNT(p.counters, CNT_OVERFLOW), 1);
            } else if (!split) {
                p.chunks[item] = ChunkItem{(int32_t)r, -1, rb[k], rb[k] + deg[k]};
            } else {
                const int64_t len = (deg[k] + nch - 1) / nch;
                const int64_t end = rb[k] + deg[k];
                p.heavy[hid] = HeavyRow{(int32_t)r, slot, nch, 0};
                for (int c = 0; c < nch; ++c) {
                    const int64_t cb = rb[k] + c * len;
                    p.chunks[item + c] = ChunkItem{(int32_t)r, slot + c, cb < end ? cb : end,
                                                   cb + len < end ? cb + len : end};
                }
            }
            hid += split;
            item += nch;
            slot += split ? nch : 0;
        }
    }
}

// Launches the degree binning over pp.N rows.  Large graphs take 2048 rows
// per block, smaller ones 1024, giving more blocks in parallel.  Measured on
// MI355X: 169K rows 12.8 -> 10.5 us with 1024; 2.1M rows 32 -> 44 us with
// 1024.
hipError_t launch_partition(const PartParams& pp, hipStream_t stream) {
    if (pp.N <= (int64_t(1) << 19)) {
        const int grid = (int)((pp.N + 4 * kBlock - 1) / (4 * kBlock));
        hipLaunchKernelGGL(gt_partition_kernel<4>, dim3(grid), dim3(kBlock), 0, stream, pp);
    } else {
        const int grid = (int)((pp.N + 8 * kBlock - 1) / (8 * kBlock));
        hipLaunchKernelGGL(gt_partition_kernel<8>, dim3(grid), dim3(kBlock), 0, stream, pp);
    }
    return hipGetLastError();
}

// Merge of the chunk partials of each heavy row, in chunk order (one
// wavefront per row; each lane owns H*D/64 consecutive accumulator floats).
// Partials are loaded kMergeBatch chunks at a time so their latencies
// overlap; the merge itself stays sequential in chunk order.
constexpr int kMergeBatch = 8;

template <typename T, int H, int D>
__global__ void __launch_bounds__(kBlock) gt_merge_kernel(MergeParams p) {
#pragma clang fp contract(off)
    constexpr int HD = H * D;
    constexpr int F = HD >= kWave ? HD / kWave : 1;
    constexpr int EB = Elt<T>::kBytes;
    const int lane = threadIdx.x & (kWave - 1);
    const int f0 = lane * F;
    const int head = f0 / D;
    const int32_t n_heavy = min(CNT(p.counters, CNT_HEAVY), p.cap_heavy);
    const int nwaves = gridDim.x * kWavesPerBlock;
    for (int hr = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; hr < n_heavy; hr += nwaves) {
        if (f0 >= HD) continue;
        const HeavyRow w = p.heavy[hr];
        float m = -INFINITY, l = 0.0f, acc[F];
#pragma unroll
        for (int f = 0; f < F; ++f) acc[f] = 0.0f;
        // a batch holds at most 64 accumulator floats per lane (wide rows take
        // fewer chunks per batch)
        constexpr int kB = 64 / F < kMergeBatch ? (64 / F > 1 ? 64 / F : 1) : kMergeBatch;
        for (int c0 = 0; c0 < w.nch; c0 += kB) {
            float2 ml[kB];
            float a[kB][F];
#pragma unroll
            for (int u = 0; u < kB; ++u) {
                const int64_t slot = w.base + (c0 + u < w.nch ? c0 + u : w.nch - 1);
                ml[u] = p.part_ml[slot * H + head];
#pragma unroll
                for (int f = 0; f < F; ++f) a[u][f] = p.part_acc[slot * HD + f0 + f];
            }
            // chunks past the row's last are merged into nothing (selects, not
            // a loop exit, so that the batch's loads stay ahead of their use)
#pragma unroll
            for (int u = 0; u < kB; ++u) {
                const bool valid = c0 + u < w.nch;
                const float mn = fmaxf(m, ml[u].x);
                const float ca = (m == mn) ? 1.0f : fast_exp2(m - mn);
                const float cb = (ml[u].x == mn) ? 1.0f : fast_exp2(ml[u].x - mn);
                const float ln = l * ca + ml[u].y * cb;
                l = valid ? ln : l;
#pragma unroll
                for (int f = 0; f < F; ++f) {
                    const float an = acc[f] * ca + a[u][f] * cb;
                    acc[f] = valid ? an : acc[f];
                }
                m = valid ? mn : m;
            }
        }
        const float inv = l > 0.0f ? 1.0f / l : 0.0f;
        if (p.lse && f0 % D == 0) p.lse[(int64_t)w.row * H + head] = lse_of(m, l);
        char* orow = p.out + (int64_t)w.row * HD * EB;
#pragma unroll
        for (int f = 0; f < F; ++f) {
            const float o = acc[f] * inv;
            if constexpr (EB == 4)
                reinterpret_cast<float*>(orow)[f0 + f] = o;
            else
                reinterpret_cast<uint16_t*>(orow)[f0 + f] = (uint16_t)bf16_rne(o);
        }
    }
}

// Clears n ints (the work-list counters at the start of a call).  A kernel
// rather than hipMemsetAsync, so that a call recorded into a HIP graph holds
// no memset node.
__global__ void __launch_bounds__(kBlock) gt_clear_kernel(int32_t* __restrict__ p, int32_t n) {
    for (int32_t i = threadIdx.x; i < n; i += kBlock) p[i] = 0;
}

__global__ void __launch_bounds__(kBlock) gt_csr_check_kernel(const int64_t* rowptr, const int32_t* colidx,
                                                            int64_t N, int64_t E, int32_t* bad) {
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    const int64_t tid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (tid == 0 && (rowptr[0] != 0 || rowptr[N] != E)) atomicOr(bad, 1);
    for (int64_t i = tid; i < N; i += stride)
        if (rowptr[i + 1] < rowptr[i]) atomicOr(bad, 1);
    for (int64_t k = tid; k < E; k += stride)
        if (colidx[k] < 0 || colidx[k] >= N) atomicOr(bad, 1);
}

// ----------------------------------------------------------------- host side

thread_local std::string t_last_error;

gt_status fail(gt_status s, const std::string& msg) {
    t_last_error = msg;
    return s;
}

gt_status hip_fail(hipError_t e, const char* what) {
    return fail(GT_ERROR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

struct Profiler {
    std::mutex mu;
    bool on = false;
    std::vector<std::array<hipEvent_t, 4>> pending;
};
Profiler& profiler() {
    static Profiler* p = new Profiler();
    return *p;
}

// The four phase events of one profiled call (when profiling is enabled):
// created by start(), recorded by mark(), handed to the profiler by commit().
// A call that fails before commit() destroys them.
struct PhaseEvents {
    std::array<hipEvent_t, 4> ev{};
    bool on = false;
    hipError_t start(hipStream_t stream) {
        Profiler& pr = profiler();
        {
            std::lock_guard<std::mutex> lk(pr.mu);
            on = pr.on;
        }
        if (!on) return hipSuccess;
        for (auto& e : ev) {
            const hipError_t he = hipEventCreate(&e);
            if (he != hipSuccess) return he;
        }
        return hipEventRecord(ev[0], stream);
    }
    void mark(int k, hipStream_t stream) {
        if (on) (void)hipEventRecord(ev[k], stream);
    }
    void commit(hipStream_t stream) {
        if (!on) return;
        (void)hipEventRecord(ev[3], stream);
        Profiler& pr = profiler();
        std::lock_guard<std::mutex> lk(pr.mu);
        pr.pending.push_back(ev);
        on = false;
    }
    ~PhaseEvents() {
        if (on)
            for (auto e : ev)
                if (e) (void)hipEventDestroy(e);
    }
};

// Workspace.  Every call takes a workspace block (degree-bin lists, partial
// states of split rows, work-list counters) for its own use and hands it back
// once its kernels are enqueued; the block is then tagged with an event
// recorded on the call's stream after those kernels.  A later call, on any
// stream, takes a free block only if its event has completed, or if it was
// last used on the same stream, and then with a device-side wait on the event
// (hipStreamWaitEvent: stream order already implies it, and it keeps a
// recycled stream handle safe); the host never waits.  Otherwise the call
// gets a new block from the library's memory pool of the device
// (hipMallocFromPoolAsync on its stream).  Blocks are not tied to streams or
// pointers, and free blocks beyond kCacheBytes per device go back to the pool
// (stream-ordered after their last use); gt_workspace_release() returns every
// free block and trims the pools.  (Freeing each call's block with
// hipFreeAsync made the host wait in every call for the previous call's
// kernels, about 485 us per call behind a 0.5 ms kernel, so the host could
// never run ahead of the device.)  While the call's stream is being captured
// into a graph, the block is allocated and freed stream-ordered instead (both
// become graph nodes), since events recorded during a capture cannot be
// queried.
constexpr int kMaxDevices = 64;
constexpr uint64_t kPoolKeepBytes = uint64_t(256) << 20;
constexpr size_t kCacheBytes = size_t(256) << 20;  // free blocks kept per device
constexpr size_t kBlockGranule = size_t(1) << 20;

struct DevicePools {
    std::once_flag once[kMaxDevices];
    hipMemPool_t pool[kMaxDevices] = {};
    hipError_t err[kMaxDevices] = {};
    std::atomic<bool> ready[kMaxDevices] = {};  // pool[dev] / err[dev] are set
};
DevicePools& device_pools() {
    static DevicePools* p = new DevicePools();
    return *p;
}

hipError_t pool_of(int dev, hipMemPool_t* out) {
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    DevicePools& dp = device_pools();
    std::call_once(dp.once[dev], [&] {
        hipMemPoolProps props;
        std::memset(&props, 0, sizeof props);
        props.allocType = hipMemAllocationTypePinned;
        props.handleTypes = hipMemHandleTypeNone;
        props.location.type = hipMemLocationTypeDevice;
        props.location.id = dev;
        hipMemPool_t pool = nullptr;
        hipError_t e = hipMemPoolCreate(&pool, &props);
        if (e == hipSuccess) {
            uint64_t keep = kPoolKeepBytes;
            e = hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
        }
        dp.pool[dev] = pool;
        dp.err[dev] = e;
        dp.ready[dev].store(true, std::memory_order_release);
    });
    *out = dp.pool[dev];
    return dp.err[dev];
}

struct WsBlock {
    char* ptr = nullptr;
    size_t bytes = 0;
    hipEvent_t ev = nullptr;       // recorded after the last user's kernels
    hipStream_t last = nullptr;    // the last user's stream
    // Forward calls keep two work-list counter sets at the start of the
    // block and use set gen % 2; each call's partition zeroes the other set
    // for the next call.  primed: set gen % 2 is zero (the last user was a
    // forward call whose partition was enqueued), so no clear is needed.
    uint32_t gen = 0;
    bool primed = false;
};

// Free blocks of one device, and the bytes of blocks that calls hold.
struct BlockCache {
    std::mutex mu;
    std::vector<WsBlock> free_blocks;
    size_t free_bytes = 0;
    size_t taken_bytes = 0;
};
BlockCache& block_cache(int dev) {
    static BlockCache* c = new BlockCache[kMaxDevices];
    return c[dev];
}

// Returns a block to the pool after its last use: ordered after the block's
// event on `stream` (the stream of the call that lets it go).
void free_block(const WsBlock& b, hipStream_t stream) {
    if (b.ev) {
        if (hipEventQuery(b.ev) != hipSuccess) (void)hipStreamWaitEvent(stream, b.ev, 0);
        (void)hipGetLastError();
        (void)hipEventDestroy(b.ev);
    }
    (void)hipFreeAsync(b.ptr, stream);
}

// One call's workspace; handed back (cached) or freed stream-ordered after
// the call's kernels when it goes out of scope (also on an error return
// after some launches).
struct CallWorkspace {
    enum Kind { NONE, CACHED, STREAM_ORDERED, SCRATCH };
    char* ptr = nullptr;
    hipStream_t stream = nullptr;
    int dev = -1;
    Kind kind = NONE;
    WsBlock block;
    bool keep_primed = false;  // set by a forward call once its partition is enqueued
    CallWorkspace() = default;
    CallWorkspace(const CallWorkspace&) = delete;
    CallWorkspace& operator=(const CallWorkspace&) = delete;
    ~CallWorkspace() {
        if (kind == STREAM_ORDERED) {
            (void)hipFreeAsync(ptr, stream);
        } else if (kind == CACHED) {
            BlockCache& c = block_cache(dev);
            if (hipEventRecord(block.ev, stream) != hipSuccess) {
                // no event, no safe reuse: free it in stream order
                (void)hipGetLastError();
                (void)hipEventDestroy(block.ev);
                block.ev = nullptr;
                (void)hipFreeAsync(block.ptr, stream);
                std::lock_guard<std::mutex> lk(c.mu);
                c.taken_bytes -= block.bytes;
                return;
            }
            block.last = stream;
            block.primed = keep_primed;
            std::vector<WsBlock> evict;
            {
                std::lock_guard<std::mutex> lk(c.mu);
                c.taken_bytes -= block.bytes;
                c.free_blocks.push_back(block);
                c.free_bytes += block.bytes;
                // over the cache bound: give back free blocks, completed ones
                // first, then the oldest
                while (c.free_bytes > kCacheBytes && !c.free_blocks.empty()) {
                    size_t k = 0;
                    for (size_t i = 0; i < c.free_blocks.size(); ++i)
                        if (hipEventQuery(c.free_blocks[i].ev) == hipSuccess) {
                            k = i;
                            break;
                        }
                    c.free_bytes -= c.free_blocks[k].bytes;
                    evict.push_back(c.free_blocks[k]);
                    c.free_blocks.erase(c.free_blocks.begin() + (std::ptrdiff_t)k);
                }
            }
            (void)hipGetLastError();
            for (const WsBlock& b : evict) free_block(b, stream);
        }
    }
};

gt_status acquire_workspace(int dev, size_t bytes, hipStream_t stream, CallWorkspace& ws) {
    hipMemPool_t pool = nullptr;
    hipError_t he = pool_of(dev, &pool);
    if (he != hipSuccess) return hip_fail(he, "workspace pool");
    ws.stream = stream;
    ws.dev = dev;
    const size_t need = (bytes + kBlockGranule - 1) / kBlockGranule * kBlockGranule;
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if ((he = hipStreamIsCapturing(stream, &cap)) != hipSuccess) return hip_fail(he, "hipStreamIsCapturing");
    const bool capturing = cap != hipStreamCaptureStatusNone;
    if (!capturing) {
        // a free block that fits: completed first, then last used on this
        // stream; the smallest such
        BlockCache& c = block_cache(dev);
        bool found = false, done = false;
        {
            std::lock_guard<std::mutex> lk(c.mu);
            size_t best = 0;
            int best_rank = 2;
            for (size_t i = 0; i < c.free_blocks.size(); ++i) {
                const WsBlock& b = c.free_blocks[i];
                if (b.bytes < need) continue;
                const hipError_t q = hipEventQuery(b.ev);
                const int rank = q == hipSuccess ? 0 : (q == hipErrorNotReady && b.last == stream) ? 1 : 2;
                if (rank < best_rank || (rank == best_rank && rank < 2 && b.bytes < c.free_blocks[best].bytes)) {
                    best = i;
                    best_rank = rank;
                }
            }
            (void)hipGetLastError();  // a query's not-ready status
            if (best_rank < 2) {
                ws.block = c.free_blocks[best];
                c.free_blocks.erase(c.free_blocks.begin() + (std::ptrdiff_t)best);
                c.free_bytes -= ws.block.bytes;
                c.taken_bytes += ws.block.bytes;
                found = true;
                done = best_rank == 0;
            }
        }
        if (found) {
            ws.kind = CallWorkspace::CACHED;
            ws.ptr = ws.block.ptr;
            if (!done && (he = hipStreamWaitEvent(stream, ws.block.ev, 0)) != hipSuccess)
                return hip_fail(he, "workspace wait");
            return GT_SUCCESS;
        }
    }
    void* p = nullptr;
    he = hipMallocFromPoolAsync(&p, capturing ? bytes : need, pool, stream);
    if (he != hipSuccess || !p) {
        (void)hipGetLastError();
        return fail(GT_ERROR_OUT_OF_MEMORY, "workspace allocation of " + std::to_string(bytes) + " bytes failed");
    }
    ws.ptr = static_cast<char*>(p);
    if (capturing) {
        ws.kind = CallWorkspace::STREAM_ORDERED;
        return GT_SUCCESS;
    }
    hipEvent_t ev = nullptr;
    if ((he = hipEventCreateWithFlags(&ev, hipEventDisableTiming)) != hipSuccess) {
        ws.kind = CallWorkspace::STREAM_ORDERED;  // freed in stream order on return
        return hip_fail(he, "workspace event");
    }
    ws.block = WsBlock{ws.ptr, need, ev, stream};
    ws.kind = CallWorkspace::CACHED;
    BlockCache& c = block_cache(dev);
    std::lock_guard<std::mutex> lk(c.mu);
    c.taken_bytes += need;
    return GT_SUCCESS;
}

// Device address of the scratch array on device `dev` (the current device),
// looked up once per device.
struct ScratchAddrs {
    std::once_flag once[kMaxDevices];
    char* ptr[kMaxDevices] = {};
    hipError_t err[kMaxDevices] = {};
};
ScratchAddrs& scratch_addrs() {
    static ScratchAddrs* s = new ScratchAddrs();
    return *s;
}

hipError_t scratch_of(int dev, char** out) {
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    ScratchAddrs& sa = scratch_addrs();
    std::call_once(sa.once[dev], [&] {
        void* p = nullptr;
        sa.err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        sa.ptr[dev] = sa.err[dev] == hipSuccess ? static_cast<char*>(p) : nullptr;
    });
    *out = sa.ptr[dev];
    if (sa.err[dev] == hipSuccess && !sa.ptr[dev]) return hipErrorInvalidSymbol;
    return sa.err[dev];
}

// The workspace of one call: from the pool, or (allocation-free entry point)
// the device's scratch array, whose size bounds the accepted problems.
gt_status call_workspace(bool noalloc, int dev, size_t bytes, hipStream_t stream, CallWorkspace& ws) {
    if (!noalloc) return acquire_workspace(dev, bytes, stream, ws);
    if (bytes > kScratchBytes)
        return fail(GT_ERROR_INVALID_VALUE, "the call needs " + std::to_string(bytes) +
                                                " bytes of workspace, more than the " + std::to_string(kScratchBytes) +
                                                "-byte scratch array of gt_attn_fwd_noalloc");
    char* p = nullptr;
    const hipError_t he = scratch_of(dev, &p);
    if (he != hipSuccess) return hip_fail(he, "hipGetSymbolAddress(scratch)");
    ws.ptr = p;
    ws.stream = stream;
    ws.kind = CallWorkspace::SCRATCH;
    return GT_SUCCESS;
}

// Zeroes `n` counter ints of a fresh workspace, in stream order.
hipError_t clear_counters(int32_t* p, int n, hipStream_t stream) {
    hipLaunchKernelGGL(gt_clear_kernel, dim3(1), dim3(kBlock), 0, stream, p, n);
    return hipGetLastError();
}

struct Args {
    const int64_t* rowptr;
    const int32_t* colidx;
    const void* Q;
    const void* K;
    const void* V;
    void* out;
    float* lse;
    int64_t N, E;
    int32_t H, D;
    float scale;
    int kind = KIND_GT;
    const float* att = nullptr;  // GATv2 attention vector
    float slope = 0.0f;          // GATv2 LeakyReLU slope
    bool noalloc = false;        // workspace from the scratch array, no allocation
};

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Capacities of the partition's lists for E entries.  Split rows have degree
// > chunk, so they number at most E/(chunk+1); front rows (degree >=
// heavy_min) at most E/heavy_min.  A split row of degree d has fewer than
// 2d/chunk chunks, so work items are at most E/heavy_min + 2E/chunk and
// partial-state slots at most 2E/chunk.  The merge kernel's grid follows the
// split-row bound.
struct PartCaps {
    int64_t heavy, items, slots;
};

PartCaps part_caps(int64_t E, int heavy_min, int chunk) {
    PartCaps c;
    c.heavy = E / ((int64_t)chunk + 1) + 1;
    c.slots = 2 * (E / chunk) + 1;
    c.items = E / heavy_min + c.slots;
    return c;
}

// Default chunk length of split rows.  A chunk is one wavefront's chain of
// dependent steps (P*U entries each, about one memory round trip, ~1 us), so
// the longest chunk bounds the call from below.  On a small graph a 1024-entry
// chunk outlasts everything else: on the arxiv-shaped power-law graph with
// fp32 4x32 features, 16K nodes took 76 us per call at 1024 against 48 us at
// 256, and 65K nodes 114 us against 95 us at 512.  The default keeps a chunk's
// steps within half the time the call's gathers take at ~7 TB/s, in multiples
// of 64, capped at 1024 (longer chunks on large graphs: default_chunk_long
// below).  With the graph-transformer forward (two gathered rows per entry)
// the arxiv-shaped 169K-node graph gets 1024; the GATv2 forward, one gathered
// row per entry, gets 768 there and 1024 from about twice its size.
double chunk_budget(int64_t E, int64_t bytes_per_entry, int entries_per_step) {
    constexpr double kGatherBytesPerSecond = 7.0e12, kStepSeconds = 1.0e-6;
    const double gather_seconds = (double)E * (double)bytes_per_entry / kGatherBytesPerSecond;
    return 0.5 * gather_seconds / kStepSeconds * entries_per_step;
}

int default_chunk(int64_t E, int64_t bytes_per_entry, int entries_per_step) {
    const double entries = chunk_budget(E, bytes_per_entry, entries_per_step);
    if (entries >= 1024.0) return 1024;
    const int64_t c = ((int64_t)entries + kWave - 1) / kWave * kWave;
    return (int)(c < kWave ? kWave : c);
}

// Chunks and front rows on large graphs (the graph-transformer forward, its
// backward and the segment reduction; the GATv2 forward keeps the rule
// above).  Where a chunk of an eighth of the gather time holds more than
// 1024 entries, chunks take that length, up to 8192; and where a wave holds
// two or more rows, only rows of at least a quarter chunk go first as front
// rows, the others being medium rows of one wavefront each.  Measured per call
// against 1024-entry chunks and a front threshold of 256: R-MAT scale 21 fp32
// 4x32 6.528 -> 6.260 ms and bf16 3.103 -> 2.936 ms, the backward on the bf16
// one 8.30 -> 7.97 ms, the 512-feature min on the fp32 one 14.45 -> 14.27 ms;
// the arxiv-shaped power-law graph at 2.1M nodes about 1 % faster; the
// lognormal-hub and SBM graphs level; graphs up to the 169K-node one keep
// their chunks.  With one row per wave (lognormal hubs, 8x64 bf16) a front
// threshold of 2048 cost 0.3-0.6 %, so those shapes keep 256.  (For the GATv2
// score the same lengths made R-MAT bf16 1.5 % slower.)
int default_chunk_long(int64_t E, int64_t bytes_per_entry, int entries_per_step) {
    const double quarter = 0.25 * chunk_budget(E, bytes_per_entry, entries_per_step);
    if (quarter <= 1024.0) return default_chunk(E, bytes_per_entry, entries_per_step);
    if (quarter >= 8192.0) return 8192;
    return (int)(((int64_t)quarter + kWave - 1) / kWave * kWave);
}

int default_front(int chunk, int rows_per_wave) {
    return rows_per_wave >= 2 && chunk / 4 > 256 ? chunk / 4 : 256;
}

// The device a call works on: the calling thread's current device.  The
// workspace, its events and the kernels' memory all belong to it, so a stream
// created on another device is refused rather than fed memory it may not be
// able to reach.  (A stream handle the runtime cannot resolve is left to the
// launch, which reports it.)
gt_status call_device(hipStream_t stream, int* dev) {
    hipError_t he = hipGetDevice(dev);
    if (he != hipSuccess) return hip_fail(he, "hipGetDevice");
    hipDevice_t sd = *dev;
    if (hipStreamGetDevice(stream, &sd) != hipSuccess) {
        (void)hipGetLastError();
        return GT_SUCCESS;
    }
    if (sd != *dev)
        return fail(GT_ERROR_INVALID_VALUE, "the stream belongs to device " + std::to_string(sd) +
                                                ", the current device is " + std::to_string(*dev));
    return GT_SUCCESS;
}

int device_cus(int dev) {
    static std::atomic<int> cache[64];
    if (dev < 0 || dev >= 64) return 256;
    if (cache[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
        cache[dev] = n;
    }
    return cache[dev];
}

template <typename T, int H, int D, int KIND>
int attn_blocks_per_cu(int dev) {
    static std::atomic<int> cache[64];
    if (dev < 0 || dev >= 64) return 4;
    if (cache[dev] == 0) {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, gt_attn_kernel<T, H, D, KIND>, kBlock, 0) != hipSuccess ||
            nb <= 0)
            nb = 4;
        cache[dev] = nb;
    }
    return cache[dev];
}

constexpr int kDefaultTileMin = 256;

template <typename T, int H, int D, int KIND>
gt_status launch(const Args& a, const gt_tuning* tu, hipStream_t stream) {
    using Gm = Geo<T, H, D>;
    // Defaults chosen by measurement on the five workload shapes (power law,
    // R-MAT, SBM, lognormal hubs): a group handles rows of up to 8 steps;
    // rows of degree >= 256 go first, split into chunks of up to 1024
    // entries, shorter ones on small graphs (default_chunk); on large graphs
    // longer chunks and, where a wave holds several rows, a higher front
    // threshold (default_chunk_long, default_front).  GATv2
    // counts its own single gather per entry but the graph-transformer step:
    // that put its chunks at the measured optimum on the arxiv-shaped graph
    // with 16K and 65K nodes (65K: 92.6 -> 77.5 us per call) and at 768
    // entries on the 169K-node one (within 1 % of 1024).  Its own half step
    // would give 384 entries there, 5.7 % slower.
    int light_max = 8 * Gm::kU;
    int chunk = KIND != KIND_GATV2
                    ? default_chunk_long(a.E, 2 * Gm::kRowBytes, Gm::kP * StepOf<T, H, D, KIND_GT>::value)
                    : default_chunk(a.E, Gm::kRowBytes, Gm::kP * StepOf<T, H, D, KIND_GT>::value);
    int heavy_min = KIND != KIND_GATV2 ? default_front(chunk, Gm::kP) : 256;
    int grid = 0;
    // Dense-tile windows (tile shapes only): on by default, for windows
    // estimated to hold at least 256 in-window entries, which a 64-row block
    // at half density holds about eight times over (measured on the SBM
    // workload; on the R-MAT one no window qualifies and the tile kernel
    // finds an empty list).
    int tile_min = kDefaultTileMin;
    if (tu) {
        if (tu->dense_tiles != 0) tile_min = tu->dense_tiles;  // < 0: off
        if (tu->light_max_deg > 0) light_max = tu->light_max_deg;
        if (tu->heavy_min_deg > 0) heavy_min = tu->heavy_min_deg;
        if (tu->chunk_edges > 0) chunk = (tu->chunk_edges + kWave - 1) / kWave * kWave;
        if (tu->grid_blocks > 0) grid = tu->grid_blocks;
    }
    if (heavy_min <= light_max) heavy_min = light_max + 1;
    constexpr bool kTileShape =
        KIND != KIND_GATV2 && std::is_same<T, bf16_tag>::value && H * D <= 128 && D % 32 == 0;
    static_assert(!kTileShape || SortedLight<T, H, D, KIND>::value,
                  "the tile path leaves its rows out of the light-row order");
    const bool tiles = kTileShape && tile_min > 0;
    if (tiles && light_max > kWinMaxDeg) light_max = kWinMaxDeg;

    int dev = 0;
    if (const gt_status ds = call_device(stream, &dev); ds != GT_SUCCESS) return ds;
    hipError_t he = hipSuccess;
    if (grid <= 0) {
        // About two light items (P rows each) per wave, between 4x and 64x the
        // number of workgroups the device holds at once: finer than one
        // resident wave of workgroups so the hardware scheduler evens out the
        // per-wave work, coarse enough to keep dispatch cheap.
        const int64_t resident = (int64_t)device_cus(dev) * attn_blocks_per_cu<T, H, D, KIND>(dev);
        const int64_t light_items = (a.N + Gm::kP - 1) / Gm::kP;
        int64_t g = light_items / (2 * kWavesPerBlock);
        if (g < 4 * resident) g = 4 * resident;
        if (g > 64 * resident) g = 64 * resident;
        const int64_t need = (light_items + kWavesPerBlock - 1) / kWavesPerBlock;
        if (g > need) g = need;
        grid = (int)(g > 0 ? g : 1);
    }
    grid = (grid + kXcds - 1) / kXcds * kXcds;

    // workspace: counters | medium rows | heavy rows | chunk items | partial (m,l) | partial acc
    const PartCaps caps = part_caps(a.E, heavy_min, chunk);
    size_t off = 0;
    const size_t o_cnt = off;      off = align_up(off + 2 * kCntSetWords * sizeof(int32_t), 256);  // two sets
    const size_t o_med = off;      off = align_up(off + (size_t)a.N * sizeof(int32_t), 256);
    const size_t o_heavy = off;    off = align_up(off + (size_t)caps.heavy * sizeof(HeavyRow), 256);
    const size_t o_chunks = off;   off = align_up(off + (size_t)caps.items * sizeof(ChunkItem), 256);
    const size_t o_ml = off;       off = align_up(off + (size_t)caps.slots * H * sizeof(float2), 256);
    const size_t o_acc = off;      off = align_up(off + (size_t)caps.slots * H * D * sizeof(float), 256);
    const size_t o_light = off;
    off = align_up(off + (!SortedLight<T, H, D, KIND>::value ? 0 : (size_t)a.N * sizeof(int32_t)), 256);
    const int64_t n_windows = (a.N + kWin - 1) / kWin;
    const size_t o_win = off;
    off = align_up(off + (tiles ? (size_t)n_windows : 0), 256);
    const size_t ws_bytes = off;

    CallWorkspace cw;
    gt_status st = call_workspace(a.noalloc, dev, ws_bytes, stream, cw);
    if (st != GT_SUCCESS) return st;
    char* ws = cw.ptr;
    // Counter sets: a cached block alternates between its two (the partition
    // zeroes the other one for the block's next call), so a block whose last
    // user was a forward call needs no clear kernel; a new block, the
    // scratch array and a captured stream clear the one set they use.
    int32_t* cnt_base = reinterpret_cast<int32_t*>(ws + o_cnt);
    const bool alternate = cw.kind == CallWorkspace::CACHED;
    int32_t* counters = cnt_base + (alternate ? (cw.block.gen & 1u) * kCntSetWords : 0);

    // (the allocation-free entry point records no profiling events: creating
    // them is a runtime allocation)
    PhaseEvents ph;
    if (!a.noalloc && (he = ph.start(stream)) != hipSuccess) return hip_fail(he, "profiling events");
    if (!(alternate && cw.block.primed) && (he = clear_counters(counters, kCntSetWords, stream)) != hipSuccess)
        return hip_fail(he, "counter clear");

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
    pp.light_list = !SortedLight<T, H, D, KIND>::value ? nullptr : reinterpret_cast<int32_t*>(ws + o_light);
    pp.step = RowState<T, H, D, KIND>::kU;
    if (tiles) {
        pp.colidx = a.colidx;
        pp.win_flags = reinterpret_cast<uint8_t*>(ws + o_win);
        pp.tile_min = tile_min;
    }
    if (alternate) pp.zero_next = cnt_base + ((cw.block.gen + 1u) & 1u) * kCntSetWords;
    if ((he = launch_partition(pp, stream)) != hipSuccess) return hip_fail(he, "partition launch");
    if (alternate) {
        ++cw.block.gen;
        cw.keep_primed = true;
    }
    ph.mark(1, stream);  // the attention phase includes the tile kernel
    if constexpr (kTileShape) {
        if (tiles) {
            TileParams tp;
            tp.rowptr = a.rowptr;
            tp.colidx = a.colidx;
            tp.Q = static_cast<const char*>(a.Q);
            tp.K = static_cast<const char*>(a.K);
            tp.V = static_cast<const char*>(a.V);
            tp.out = static_cast<char*>(a.out);
            tp.lse = a.lse;
            tp.N = a.N;
            tp.c = a.scale * 1.4426950408889634f;
            tp.light_max = light_max;
            tp.min_entries = tile_min;
            tp.win_flags = pp.win_flags;
            tp.counters = counters;
            hipLaunchKernelGGL((gt_tile_kernel<H, D, KIND>), dim3((unsigned)n_windows), dim3(kBlock), 0, stream, tp);
            if ((he = hipGetLastError()) != hipSuccess) return hip_fail(he, "tile launch");
        }
    }

    AttnParams ap;
    ap.rowptr = a.rowptr;
    ap.colidx = a.colidx;
    ap.Q = static_cast<const char*>(a.Q);
    ap.K = static_cast<const char*>(a.K);
    ap.V = static_cast<const char*>(a.V);
    ap.out = static_cast<char*>(a.out);
    ap.lse = a.lse;
    ap.N = a.N;
    ap.c = (KIND != KIND_GATV2 ? a.scale : 1.0f) * 1.4426950408889634f;
    ap.att = a.att;
    ap.slope = a.slope;
    ap.light_max = light_max;
    ap.cap_items = (int32_t)caps.items;
    ap.counters = counters;
    ap.med_list = pp.med_list;
    ap.chunks = pp.chunks;
    ap.part_acc = reinterpret_cast<float*>(ws + o_acc);
    ap.part_ml = reinterpret_cast<float2*>(ws + o_ml);
    ap.light_list = pp.light_list;
    hipLaunchKernelGGL((gt_attn_kernel<T, H, D, KIND>), dim3(grid), dim3(kBlock), 0, stream, ap);
    if ((he = hipGetLastError()) != hipSuccess) return hip_fail(he, "attention launch");
    ph.mark(2, stream);

    MergeParams mp;
    mp.cap_heavy = (int32_t)caps.heavy;
    mp.counters = counters;
    mp.heavy = pp.heavy;
    mp.part_acc = ap.part_acc;
    mp.part_ml = ap.part_ml;
    mp.out = ap.out;
    mp.lse = a.lse;
    int merge_grid = (int)((caps.heavy + kWavesPerBlock - 1) / kWavesPerBlock);
    const int merge_cap = device_cus(dev) * 8;
    if (merge_grid > merge_cap) merge_grid = merge_cap;
    if (merge_grid < 1) merge_grid = 1;
    hipLaunchKernelGGL((gt_merge_kernel<T, H, D>), dim3(merge_grid), dim3(kBlock), 0, stream, mp);
    if ((he = hipGetLastError()) != hipSuccess) return hip_fail(he, "merge launch");
    ph.commit(stream);
    return GT_SUCCESS;
}

using LaunchFn = gt_status (*)(const Args&, const gt_tuning*, hipStream_t);

template <typename T, int KIND>
LaunchFn pick_hd(int32_t H, int32_t D) {
#define GT_CASE(h, d) \
    if (H == h && D == d) return &launch<T, h, d, KIND>;
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

bool overlaps(const void* a, size_t an, const void* b, size_t bn) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + bn && y < x + an;
}

// Tuning fields are counts of entries, rows or workgroups: positive values
// beyond kTuningMax (about 2^31 - 2^16) would overflow the partition's
// rounding and comparisons, so they are refused.
constexpr int32_t kTuningMax = INT32_MAX - (1 << 16);

gt_status check_tuning(const gt_tuning* tu) {
    if (!tu) return GT_SUCCESS;
    const int32_t f[] = {tu->light_max_deg, tu->heavy_min_deg, tu->chunk_edges, tu->grid_blocks, tu->dense_tiles};
    for (int32_t v : f)
        if (v > kTuningMax)
            return fail(GT_ERROR_INVALID_VALUE, "a tuning field exceeds " + std::to_string(kTuningMax));
    return GT_SUCCESS;
}

gt_status run(gt_dtype dtype, const Args& a, const gt_tuning* tu, hipStream_t stream) {
    t_last_error.clear();
    if (check_tuning(tu) != GT_SUCCESS) return GT_ERROR_INVALID_VALUE;
    if (dtype != GT_DTYPE_F32 && dtype != GT_DTYPE_BF16) return fail(GT_ERROR_NOT_SUPPORTED, "unknown dtype");
    if (a.N < 0 || a.N >= (int64_t(1) << 31)) return fail(GT_ERROR_INVALID_VALUE, "N must be in [0, 2^31)");
    if (a.E < 0 || a.E >= (int64_t(1) << 31)) return fail(GT_ERROR_INVALID_VALUE, "E must be in [0, 2^31)");
    if (a.H < 1 || a.D < 1) return fail(GT_ERROR_INVALID_VALUE, "H and D must be positive");
    if (!std::isfinite(a.scale)) return fail(GT_ERROR_INVALID_VALUE, "scale must be finite");
    if (a.kind == KIND_GATV2 && !std::isfinite(a.slope)) return fail(GT_ERROR_INVALID_VALUE, "slope must be finite");
    LaunchFn fn;
    if (a.kind == KIND_GATV2)
        fn = dtype == GT_DTYPE_F32 ? pick_hd<float, KIND_GATV2>(a.H, a.D) : pick_hd<bf16_tag, KIND_GATV2>(a.H, a.D);
    else
        fn = dtype == GT_DTYPE_F32 ? pick_hd<float, KIND_GT>(a.H, a.D)
             : (tu && tu->bf16_weights) ? pick_hd<bf16_tag, KIND_GT_BF16W>(a.H, a.D)
                                        : pick_hd<bf16_tag, KIND_GT>(a.H, a.D);
    if (!fn)
        return fail(GT_ERROR_NOT_SUPPORTED, "unsupported (H, D) = (" + std::to_string(a.H) + ", " +
                                                std::to_string(a.D) + "); H in {1,2,4,8} with D in {32,64,128,256}, or bf16 D = 512 with H in {1,2,4}");
    if (a.N == 0) return GT_SUCCESS;
    if (!a.rowptr) return fail(GT_ERROR_INVALID_VALUE, "rowptr is null");
    if (a.E > 0 && !a.colidx) return fail(GT_ERROR_INVALID_VALUE, "colidx is null");
    if (!a.Q || !a.K || !a.V || !a.out) return fail(GT_ERROR_INVALID_VALUE, "Q, K, V and out (L, R and out) must be non-null");
    for (const void* ptr : {a.Q, a.K, a.V, static_cast<const void*>(a.out)})
        if (reinterpret_cast<uintptr_t>(ptr) % 16 != 0)
            return fail(GT_ERROR_INVALID_VALUE, "Q, K, V and out (L, R and out) must be 16-byte aligned");
    const size_t bytes = (size_t)a.N * a.H * a.D * (dtype == GT_DTYPE_F32 ? 4 : 2);
    for (const void* in : {a.Q, a.K, a.V})
        if (overlaps(a.out, bytes, in, bytes)) return fail(GT_ERROR_INVALID_VALUE, "out overlaps Q, K or V (L or R)");
    if (a.lse) {
        const size_t lb = (size_t)a.N * a.H * sizeof(float);
        if (reinterpret_cast<uintptr_t>(a.lse) % 4 != 0) return fail(GT_ERROR_INVALID_VALUE, "lse must be 4-byte aligned");
        for (const void* o : {a.Q, a.K, a.V, static_cast<const void*>(a.out)})
            if (overlaps(a.lse, lb, o, bytes)) return fail(GT_ERROR_INVALID_VALUE, "lse overlaps Q, K, V or out");
    }
    if (a.kind == KIND_GATV2) {
        const size_t ab = (size_t)a.H * a.D * sizeof(float);
        if (!a.att || reinterpret_cast<uintptr_t>(a.att) % 16 != 0)
            return fail(GT_ERROR_INVALID_VALUE, "att must be non-null and 16-byte aligned");
        if (overlaps(a.out, bytes, a.att, ab) || (a.lse && overlaps(a.lse, (size_t)a.N * a.H * sizeof(float), a.att, ab)))
            return fail(GT_ERROR_INVALID_VALUE, "out or lse overlaps att");
    }
    return fn(a, tu, stream);
}

#include "gt_bwd.hpp"

gt_status run_bwd(gt_dtype dtype, const BwdArgs& a, hipStream_t stream) {
    t_last_error.clear();
    if (dtype != GT_DTYPE_F32 && dtype != GT_DTYPE_BF16) return fail(GT_ERROR_NOT_SUPPORTED, "unknown dtype");
    if (a.N < 0 || a.N >= (int64_t(1) << 31)) return fail(GT_ERROR_INVALID_VALUE, "N must be in [0, 2^31)");
    if (a.E < 0 || a.E >= (int64_t(1) << 31)) return fail(GT_ERROR_INVALID_VALUE, "E must be in [0, 2^31)");
    if (a.H < 1 || a.D < 1) return fail(GT_ERROR_INVALID_VALUE, "H and D must be positive");
    if (!std::isfinite(a.scale)) return fail(GT_ERROR_INVALID_VALUE, "scale must be finite");
    BwdFn fn = dtype == GT_DTYPE_F32 ? pick_bwd<float>(a.H, a.D) : pick_bwd<bf16_tag>(a.H, a.D);
    if (!fn)
        return fail(GT_ERROR_NOT_SUPPORTED, "unsupported (H, D) = (" + std::to_string(a.H) + ", " +
                                                std::to_string(a.D) + "); H in {1,2,4,8} with D in {32,64,128,256}, or bf16 D = 512 with H in {1,2,4}");
    if (a.N == 0) return GT_SUCCESS;
    if (!a.rowptr || !a.rowptr_t) return fail(GT_ERROR_INVALID_VALUE, "rowptr or rowptr_t is null");
    if (a.E > 0 && (!a.colidx || !a.colidx_t)) return fail(GT_ERROR_INVALID_VALUE, "colidx or colidx_t is null");
    const void* ins[] = {a.Q, a.K, a.V, a.O, a.dO};
    const void* outs[] = {a.dQ, a.dK, a.dV};
    for (const void* ptr : ins)
        if (!ptr || reinterpret_cast<uintptr_t>(ptr) % 16 != 0)
            return fail(GT_ERROR_INVALID_VALUE, "Q, K, V, out and dout must be non-null and 16-byte aligned");
    for (const void* ptr : outs)
        if (!ptr || reinterpret_cast<uintptr_t>(ptr) % 16 != 0)
            return fail(GT_ERROR_INVALID_VALUE, "dQ, dK and dV must be non-null and 16-byte aligned");
    if (!a.lse || reinterpret_cast<uintptr_t>(a.lse) % 4 != 0)
        return fail(GT_ERROR_INVALID_VALUE, "lse must be non-null and 4-byte aligned");
    const size_t bytes = (size_t)a.N * a.H * a.D * (dtype == GT_DTYPE_F32 ? 4 : 2);
    for (int g = 0; g < 3; ++g) {
        for (const void* in : ins)
            if (overlaps(outs[g], bytes, in, bytes)) return fail(GT_ERROR_INVALID_VALUE, "a gradient overlaps an input");
        if (overlaps(outs[g], bytes, a.lse, (size_t)a.N * a.H * sizeof(float)))
            return fail(GT_ERROR_INVALID_VALUE, "a gradient overlaps lse");
        // distinct gradients, also when two are the same pointer
        for (int g2 = g + 1; g2 < 3; ++g2)
            if (overlaps(outs[g], bytes, outs[g2], bytes)) return fail(GT_ERROR_INVALID_VALUE, "gradients overlap");
    }
    return fn(a, stream);
}

#include "gt_reduce.hpp"

gt_status run_reduce(gt_dtype dtype, int op, const ReduceArgs& a0, const gt_tuning* tu, hipStream_t stream) {
    t_last_error.clear();
    if (dtype != GT_DTYPE_F32 && dtype != GT_DTYPE_BF16) return fail(GT_ERROR_NOT_SUPPORTED, "unknown dtype");
    if (op != GT_REDUCE_MIN && op != GT_REDUCE_MAX) return fail(GT_ERROR_NOT_SUPPORTED, "unknown reduce op");
    if (check_tuning(tu) != GT_SUCCESS) return GT_ERROR_INVALID_VALUE;
    if (a0.N < 0 || a0.N >= (int64_t(1) << 31)) return fail(GT_ERROR_INVALID_VALUE, "N must be in [0, 2^31)");
    if (a0.E < 0 || a0.E >= (int64_t(1) << 31)) return fail(GT_ERROR_INVALID_VALUE, "E must be in [0, 2^31)");
    if (a0.F < 1) return fail(GT_ERROR_INVALID_VALUE, "F must be positive");
    ReduceFn fn = dtype == GT_DTYPE_F32 ? pick_reduce<float>(a0.F) : pick_reduce<bf16_tag>(a0.F);
    if (!fn)
        return fail(GT_ERROR_NOT_SUPPORTED, "unsupported F = " + std::to_string(a0.F) +
                                                "; rows of 64 B to 4 KiB in powers of two (fp32 F in {16..1024}, "
                                                "bf16 F in {32..2048})");
    if (a0.N == 0) return GT_SUCCESS;
    if (!a0.rowptr) return fail(GT_ERROR_INVALID_VALUE, "rowptr is null");
    if (a0.E > 0 && !a0.colidx) return fail(GT_ERROR_INVALID_VALUE, "colidx is null");
    if (!a0.X || !a0.out) return fail(GT_ERROR_INVALID_VALUE, "X and out must be non-null");
    for (const void* ptr : {a0.X, static_cast<const void*>(a0.out), static_cast<const void*>(a0.arg)})
        if (reinterpret_cast<uintptr_t>(ptr) % 16 != 0)
            return fail(GT_ERROR_INVALID_VALUE, "X, out and arg must be 16-byte aligned");
    const size_t bytes = (size_t)a0.N * a0.F * (dtype == GT_DTYPE_F32 ? 4 : 2);
    const size_t abytes = (size_t)a0.N * a0.F * sizeof(int32_t);
    if (overlaps(a0.out, bytes, a0.X, bytes)) return fail(GT_ERROR_INVALID_VALUE, "out overlaps X");
    if (a0.arg && (overlaps(a0.arg, abytes, a0.X, bytes) || overlaps(a0.arg, abytes, a0.out, bytes)))
        return fail(GT_ERROR_INVALID_VALUE, "arg overlaps X or out");
    ReduceArgs a = a0;
    a.flip = op == GT_REDUCE_MAX ? 0xFFFFFFFFu : 0u;
    return fn(a, tu, stream);
}

#include "gt_study.hpp"

gt_status run_dot_aggr(const int64_t* rowptr, const int32_t* colidx, const float* X, float* out, int64_t N,
                       int64_t E, int32_t F, int32_t mapping, int32_t load_bytes, hipStream_t stream) {
    t_last_error.clear();
    if (N < 0 || N >= (int64_t(1) << 31)) return fail(GT_ERROR_INVALID_VALUE, "N must be in [0, 2^31)");
    if (E < 0 || E >= (int64_t(1) << 31)) return fail(GT_ERROR_INVALID_VALUE, "E must be in [0, 2^31)");
    DotFn fn = pick_dot(mapping, load_bytes, F);
    if (!fn)
        return fail(GT_ERROR_NOT_SUPPORTED, "unsupported dot-aggr variant: mapping in {0, 1}, load_bytes in "
                                            "{4, 16}, F in {32, 64, 128, 256, 512}");
    if (N == 0) return GT_SUCCESS;
    if (!rowptr || (E > 0 && !colidx) || !X || !out) return fail(GT_ERROR_INVALID_VALUE, "null pointer");
    if (reinterpret_cast<uintptr_t>(X) % 16 != 0 || reinterpret_cast<uintptr_t>(out) % 4 != 0)
        return fail(GT_ERROR_INVALID_VALUE, "X must be 16-byte and out 4-byte aligned");
    if (overlaps(out, (size_t)N * sizeof(float), X, (size_t)N * F * sizeof(float)))
        return fail(GT_ERROR_INVALID_VALUE, "out overlaps X");
    DotParams dp{rowptr, colidx, X, out, N};
    const int64_t blocks = (N + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL(fn, dim3((unsigned)blocks), dim3(kBlock), 0, stream, dp);
    const hipError_t he = hipGetLastError();
    if (he != hipSuccess) return hip_fail(he, "dot-aggr launch");
    return GT_SUCCESS;
}

}  // namespace

extern "C" {

gt_status gt_attn_fwd(const int64_t* rowptr, const int32_t* colidx, const float* Q, const float* K,
                      const float* V, float* out, int64_t N, int64_t E, int32_t H, int32_t D, float scale,
                      hipStream_t stream) {
    return run(GT_DTYPE_F32, Args{rowptr, colidx, Q, K, V, out, nullptr, N, E, H, D, scale}, nullptr, stream);
}

gt_status gt_attn_fwd_bf16(const int64_t* rowptr, const int32_t* colidx, const uint16_t* Q, const uint16_t* K,
                           const uint16_t* V, uint16_t* out, int64_t N, int64_t E, int32_t H, int32_t D,
                           float scale, hipStream_t stream) {
    return run(GT_DTYPE_BF16, Args{rowptr, colidx, Q, K, V, out, nullptr, N, E, H, D, scale}, nullptr, stream);
}

gt_status gt_attn_fwd_ex(gt_dtype dtype, const int64_t* rowptr, const int32_t* colidx, const void* Q,
                         const void* K, const void* V, void* out, float* lse, int64_t N, int64_t E, int32_t H,
                         int32_t D, float scale, const gt_tuning* tuning, hipStream_t stream) {
    return run(dtype, Args{rowptr, colidx, Q, K, V, out, lse, N, E, H, D, scale}, tuning, stream);
}

gt_status gt_attn_fwd_noalloc(gt_dtype dtype, const int64_t* rowptr, const int32_t* colidx, const void* Q,
                              const void* K, const void* V, void* out, float* lse, int64_t N, int64_t E, int32_t H,
                              int32_t D, float scale, const gt_tuning* tuning, hipStream_t stream) {
    Args a{rowptr, colidx, Q, K, V, out, lse, N, E, H, D, scale};
    a.noalloc = true;
    return run(dtype, a, tuning, stream);
}

gt_status gt_gatv2_fwd(gt_dtype dtype, const int64_t* rowptr, const int32_t* colidx, const void* L, const void* R,
                       const float* att, float slope, void* out, float* lse, int64_t N, int64_t E, int32_t H,
                       int32_t D, const gt_tuning* tuning, hipStream_t stream) {
    Args a{rowptr, colidx, L, R, R, out, lse, N, E, H, D, 1.0f};
    a.kind = KIND_GATV2;
    a.att = att;
    a.slope = slope;
    return run(dtype, a, tuning, stream);
}

gt_status gt_attn_bwd(gt_dtype dtype, const int64_t* rowptr, const int32_t* colidx, const int64_t* rowptr_t,
                      const int32_t* colidx_t, const void* Q, const void* K, const void* V, const void* out,
                      const void* dout, const float* lse, void* dQ, void* dK, void* dV, int64_t N, int64_t E,
                      int32_t H, int32_t D, float scale, hipStream_t stream) {
    return run_bwd(dtype,
                   BwdArgs{rowptr, colidx, rowptr_t, colidx_t, Q, K, V, out, dout, lse, dQ, dK, dV, N, E, H, D, scale},
                   stream);
}

gt_status gt_segment_reduce(gt_dtype dtype, gt_reduce_op op, const int64_t* rowptr, const int32_t* colidx,
                            const void* X, void* out, int32_t* arg, int64_t N, int64_t E, int32_t F,
                            const gt_tuning* tuning, hipStream_t stream) {
    return run_reduce(dtype, (int)op, ReduceArgs{rowptr, colidx, X, out, arg, N, E, F, 0u}, tuning, stream);
}

gt_status gt_dot_aggr(const int64_t* rowptr, const int32_t* colidx, const float* X, float* out, int64_t N,
                      int64_t E, int32_t F, int32_t mapping, int32_t load_bytes, hipStream_t stream) {
    return run_dot_aggr(rowptr, colidx, X, out, N, E, F, mapping, load_bytes, stream);
}

gt_status gt_csr_validate(const int64_t* rowptr, const int32_t* colidx, int64_t N, int64_t E, int32_t* valid,
                          hipStream_t stream) {
    t_last_error.clear();
    if (!valid) return fail(GT_ERROR_INVALID_VALUE, "valid is null");
    *valid = 0;
    if (N < 0 || E < 0 || E >= (int64_t(1) << 31)) return fail(GT_ERROR_INVALID_VALUE, "bad N or E");
    if (!rowptr || (E > 0 && !colidx)) return fail(GT_ERROR_INVALID_VALUE, "null CSR pointer");
    int32_t* bad = nullptr;
    hipError_t he = hipMallocAsync(reinterpret_cast<void**>(&bad), sizeof(int32_t), stream);
    if (he != hipSuccess) return fail(GT_ERROR_OUT_OF_MEMORY, "flag allocation failed");
    // the flag is freed (stream-ordered) on every path once it was allocated
    auto failed = [&](hipError_t e, const char* what) {
        (void)hipFreeAsync(bad, stream);
        return hip_fail(e, what);
    };
    if ((he = hipMemsetAsync(bad, 0, sizeof(int32_t), stream)) != hipSuccess) return failed(he, "hipMemsetAsync");
    const int64_t work = N > E ? N : E;
    int grid = (int)((work + kBlock - 1) / kBlock);
    if (grid > 4096) grid = 4096;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(gt_csr_check_kernel, dim3(grid), dim3(kBlock), 0, stream, rowptr, colidx, N, E, bad);
    if ((he = hipGetLastError()) != hipSuccess) return failed(he, "validate launch");
    int32_t h_bad = 1;
    if ((he = hipMemcpyAsync(&h_bad, bad, sizeof(int32_t), hipMemcpyDeviceToHost, stream)) != hipSuccess)
        return failed(he, "hipMemcpyAsync");
    (void)hipFreeAsync(bad, stream);
    if ((he = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(he, "hipStreamSynchronize");
    *valid = h_bad == 0 ? 1 : 0;
    return GT_SUCCESS;
}

const char* gt_status_string(gt_status s) {
    switch (s) {
        case GT_SUCCESS: return "success";
        case GT_ERROR_INVALID_VALUE: return "invalid value";
        case GT_ERROR_NOT_SUPPORTED: return "not supported";
        case GT_ERROR_OUT_OF_MEMORY: return "out of memory";
        case GT_ERROR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

const char* gt_last_error_message(void) { return t_last_error.c_str(); }

gt_status gt_profile_enable(int32_t enable) {
    Profiler& pr = profiler();
    std::lock_guard<std::mutex> lk(pr.mu);
    for (auto& ev : pr.pending) {
        (void)hipEventSynchronize(ev[3]);
        for (auto e : ev) (void)hipEventDestroy(e);
    }
    pr.pending.clear();
    pr.on = enable != 0;
    return GT_SUCCESS;
}

gt_status gt_profile_collect(double ms[3], int64_t* calls) {
    t_last_error.clear();
    if (!ms || !calls) return fail(GT_ERROR_INVALID_VALUE, "null output");
    Profiler& pr = profiler();
    std::lock_guard<std::mutex> lk(pr.mu);
    ms[0] = ms[1] = ms[2] = 0.0;
    *calls = 0;
    gt_status st = GT_SUCCESS;
    for (auto& ev : pr.pending) {
        hipError_t he = hipEventSynchronize(ev[3]);
        if (he != hipSuccess) {
            st = hip_fail(he, "hipEventSynchronize");
        } else {
            for (int k = 0; k < 3; ++k) {
                float t = 0.0f;
                if (hipEventElapsedTime(&t, ev[k], ev[k + 1]) == hipSuccess) ms[k] += t;
            }
            ++*calls;
        }
        for (auto e : ev) (void)hipEventDestroy(e);
    }
    pr.pending.clear();
    return st;
}

gt_status gt_workspace_pool_stats(int32_t device, uint64_t* reserved_bytes, uint64_t* used_bytes) {
    t_last_error.clear();
    if (!reserved_bytes || !used_bytes) return fail(GT_ERROR_INVALID_VALUE, "null output");
    *reserved_bytes = 0;
    *used_bytes = 0;
    if (device < 0 || device >= kMaxDevices) return fail(GT_ERROR_INVALID_VALUE, "device out of range");
    DevicePools& dp = device_pools();
    if (!dp.ready[device].load(std::memory_order_acquire) || !dp.pool[device]) return GT_SUCCESS;
    uint64_t r = 0;
    const hipError_t he = hipMemPoolGetAttribute(dp.pool[device], hipMemPoolAttrReservedMemCurrent, &r);
    if (he != hipSuccess) return hip_fail(he, "hipMemPoolGetAttribute");
    BlockCache& c = block_cache(device);
    std::lock_guard<std::mutex> lk(c.mu);
    *reserved_bytes = r;
    *used_bytes = c.taken_bytes;
    return GT_SUCCESS;
}

gt_status gt_workspace_release(void) {
    t_last_error.clear();
    DevicePools& dp = device_pools();
    gt_status st = GT_SUCCESS;
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) cur = -1;
    for (int dev = 0; dev < kMaxDevices; ++dev) {
        // a device's pool is created by its first call; devices without one
        // are skipped
        if (!dp.ready[dev].load(std::memory_order_acquire)) continue;
        hipMemPool_t pool = dp.pool[dev];
        if (!pool) continue;
        std::vector<WsBlock> blocks;
        {
            BlockCache& c = block_cache(dev);
            std::lock_guard<std::mutex> lk(c.mu);
            blocks.swap(c.free_blocks);
            c.free_bytes = 0;
        }
        hipError_t he = hipSetDevice(dev);
        // each free block after its last use, then the pool down to nothing
        for (const WsBlock& b : blocks) {
            if (he == hipSuccess) he = hipEventSynchronize(b.ev);
            (void)hipEventDestroy(b.ev);
            if (he == hipSuccess) he = hipFreeAsync(b.ptr, nullptr);
        }
        if (he == hipSuccess) he = hipStreamSynchronize(nullptr);
        if (he == hipSuccess) he = hipMemPoolTrimTo(pool, 0);
        if (he != hipSuccess) st = hip_fail(he, "returning workspace of a device");
    }
    if (cur >= 0) (void)hipSetDevice(cur);
    return st;
}

}  // extern "C"
