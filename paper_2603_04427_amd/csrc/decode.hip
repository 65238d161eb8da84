// Thin-key decode attention for gfx950: split-K over the cached context.
//
// One decode step reads every cached key row (r entries) and value row (d_v
// entries) once; that stream dominates the step's memory traffic, which is why
// decode is bandwidth-bound (Sec. 4.2, Eq. 10) and why thin keys cut its cost
// by (r + d_v) / (2 d_head) (Eq. 8-9). The kernels here are built around that:
//
//  * Grouped-query packing: a workgroup serves all HG query heads that share a
//    KV head, so each K/V byte crosses HBM once for HG heads.
//  * Each wave streams 32- or 64-token chunks with 16-byte non-temporal loads
//    per lane (each byte is read once per step), all of a chunk's K and V
//    loads issued before any arithmetic: key rows tile the lanes (LPT lanes
//    per row, one 16-byte slice each), value rows likewise.
//    The waves of a workgroup take consecutive chunks (one round), and the
//    splits of a (sequence, head group) take the rounds in turn, so together
//    they read one contiguous stream of each cache rather than n_split
//    separate ones.
//  * Scores: per-lane partial dot products over the lane's slice of r (the
//    query kept as exact bf16 pairs), reduced across the LPT lanes of a row
//    with DPP. One fp32 multiply by the softmax scale times log2(e) (and, for
//    quantised keys, the token's key scale) turns the reduced dot product into
//    a log2-domain logit, so the softmax uses exp2 directly.
//  * Online softmax per head: each score is exponentiated once, by the lane
//    that owns its head, against a lazy reference maximum that moves only when
//    a score exceeds it by more than 8 in log2 units, a factor of 256 (a wave
//    ballot, then a cross-lane reduction, almost never after a stream's first
//    chunk); probabilities go through a small per-wave LDS table to the lanes
//    that own the value columns.
//  * The waves of a workgroup merge their (max, sum, output) triples in LDS
//    and write one partial per (sequence, head, split). The last workgroup of a
//    (sequence, head group) to finish - found with an agent-scope counter in the
//    workspace, which it resets to zero - merges the splits with the log-sum-exp
//    rule and writes bf16, so one call is one kernel launch.
#include "tk_device.hpp"
#include "tk_internal.hpp"

#include <math.h>

#include <mutex>
#include <type_traits>

#ifndef TK_DECODE_TARGET_GROUPS
#define TK_DECODE_TARGET_GROUPS 256
#endif

namespace tk {

// Waves per workgroup, each streaming its own chunks: 4, or 8 when each wave
// would otherwise get at most four chunks of its split (short streams, where
// latency rather than bandwidth sets the time).
constexpr int kDecodeWavesLong = 4;
constexpr int kDecodeWavesShort = 8;
constexpr int kShortRounds = 4;
constexpr int kMaxSplits = 1024;
constexpr size_t kCounterRegionBytes = 2 * TK_DECODE_TARGET_GROUPS * sizeof(unsigned);
static_assert(kCounterRegionBytes % 256 == 0, "the partials after the counters stay 256-byte aligned");

// Agent-scope relaxed atomic accesses (sc1 on gfx950): coherent across XCDs.
__device__ __forceinline__ void store_coherent(float* p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_coherent(const float* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Raw buffer descriptor over `bytes` bytes at `base` (gfx9 data format word):
// loads at offsets >= bytes return zero instead of touching memory.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}
// Cache policy of the cache stream's loads: the non-temporal bit (nt), the
// hint that a line has no temporal reuse. Every K/V byte of a step is read
// exactly once, so nothing is lost by not keeping the lines, and with the hint
// the same loads run about a tenth faster (the results are bitwise the same).
constexpr int kStreamPolicy = 2;
__device__ __forceinline__ uint4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kStreamPolicy);
    return make_uint4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ uint2 buffer_load8(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, kStreamPolicy);
    return make_uint2(v[0], v[1]);
}
__device__ __forceinline__ uint32_t buffer_load4(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, kStreamPolicy);
}
// A wave-uniform 32-bit load through the scalar cache (its own counter, so
// waiting for it does not wait for the vector loads in flight).
__device__ __forceinline__ int load_uniform(const int32_t* p) {
    return *(const __attribute__((address_space(4))) int32_t*)p;
}

// Wait until this thread's outstanding global stores have completed.
__device__ __forceinline__ void wait_stores() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

template <int KF>
struct KeyRow {
    static constexpr bool SCALED = KF != kKeyBF16;
    static constexpr int SLICE = KF == kKeyInt4 ? 8 : 16;  // bytes of a key row per lane (one load)
    static constexpr int EPL = KF == kKeyBF16 ? 8 : 16;    // key entries per lane slice
    template <int R>
    static constexpr int bytes() { return KF == kKeyBF16 ? 2 * R : (KF == kKeyE4M3 ? R : R / 2); }
};

template <int R, int DV, int HG, int KF, int CH>
struct DecodeShape {
    using KR = KeyRow<KF>;
    static constexpr int ROWB = KR::template bytes<R>();  // bytes per key row
    static constexpr int LPT = ROWB / KR::SLICE;          // lanes per key row (one slice each)
    static constexpr int EPL = KR::EPL;                   // key entries per lane slice
    static constexpr int QW = EPL / 2;                    // packed bf16 query dwords per head and lane
    static constexpr int TPK = 64 / LPT;       // key rows per wave-wide load
    static constexpr int KL = CH / TPK;        // key loads per chunk
    static constexpr int LPV = DV * 2 / 16;    // lanes per value row
    static constexpr int TPV = 64 / LPV;       // value rows per wave-wide load
    static constexpr int VL = CH / TPV;        // value loads per chunk (even)
    static_assert(LPT >= 1 && LPT <= 16 && (LPV == 8 || LPV == 16), "unsupported shape");
    static_assert(KL >= 1 && VL >= 2 && VL % 2 == 0, "chunk too short for this row width");
};

// Tokens per wave iteration, and whether the next chunk's loads are issued
// before the current chunk is processed (two register buffers). Chosen so the
// buffers fit the 256-register budget of two waves per SIMD: 32-token chunks
// double-buffered where a chunk would otherwise need too many registers.
template <int R, int DV, int HG, int KF>
struct DecodeSchedule {
    using KR = KeyRow<KF>;
    static constexpr int LPT = KR::template bytes<R>() / KR::SLICE;
    static constexpr int kRegs64 = KR::template bytes<R>() / 4 + DV / 2;  // one 64-token buffer
    static constexpr int kBase = HG * 8 + HG * (KR::EPL / 2) + 2 * HG + 48 + (KF == kKeyInt4 ? HG : 0);
    static constexpr bool kFits64 = kBase + 2 * kRegs64 + HG * LPT <= 200;
    static constexpr bool kShort = !kFits64 && 64 / LPT <= 32;
    static constexpr int CH = kShort ? 32 : 64;
    static constexpr bool PIPE = kFits64 || kBase + kRegs64 + HG * LPT <= 200;
};

// One chunk of CH tokens as this lane holds it.
template <int R, int DV, int HG, int KF, int CH>
struct Chunk {
    using S = DecodeShape<R, DV, HG, KF, CH>;
    using KVec = typename std::conditional<KF == kKeyInt4, uint2, uint4>::type;
    KVec k[S::KL];
    float ks[KeyRow<KF>::SCALED ? S::KL : 1];
    uint4 v[S::VL];
    int nvalid;  // tokens of the chunk inside the context (0: skip, bad page)
};

// Issues the loads of the CH-token chunk starting at ts through raw buffer
// descriptors bounded to the rows this call may read (rows at or beyond
// `avail` come back as zeros from the hardware range check): one 32-bit offset
// per lane, a wave-uniform base, constant offsets per load, no branches.
// Returns false (and loads nothing) for a block-table entry outside
// [0, num_blocks).
template <int R, int DV, int HG, int KF, int CH, bool PAGED>
__device__ __forceinline__ bool load_chunk(Chunk<R, DV, HG, KF, CH>& c, const DecodeParams& p, int b, int g, int ts,
                                           int avail, int lane) {
    using S = DecodeShape<R, DV, HG, KF, CH>;
    const int nrows = avail - ts < CH ? avail - ts : CH;
    size_t row0;
    if constexpr (PAGED) {
        const int blk = load_uniform(p.block_table + (size_t)b * p.mb + (ts >> p.bs_log2));
        if (blk < 0 || blk >= p.num_blocks) {  // never dereference a bad entry
            c.nvalid = 0;
            return false;
        }
        row0 = (((size_t)blk * p.Hkv + g) << p.bs_log2) + (ts & ((1 << p.bs_log2) - 1));
    } else {
        row0 = ((size_t)b * p.Hkv + g) * p.max_ctx + ts;
    }
    c.nvalid = CH;  // refined against the context length when processed
    const int kgrp = lane / S::LPT, kpart = lane % S::LPT;
    const int vgrp = lane / S::LPV, vpart = lane % S::LPV;
    const auto kr = make_rsrc(p.k + row0 * S::ROWB, (uint32_t)(nrows * S::ROWB));
    const auto vr = make_rsrc(p.v + row0 * DV, (uint32_t)(nrows * DV * 2));
    const uint32_t koff = (uint32_t)(kgrp * S::ROWB + kpart * KeyRow<KF>::SLICE);
    const uint32_t voff = (uint32_t)((vgrp * DV + vpart * 8) * 2);
#pragma unroll
    for (int j = 0; j < S::KL; ++j) {
        if constexpr (KF == kKeyInt4)
            c.k[j] = buffer_load8(kr, koff, j * S::TPK * S::ROWB);
        else
            c.k[j] = buffer_load16(kr, koff, j * S::TPK * S::ROWB);
    }
    if constexpr (KeyRow<KF>::SCALED) {
        const auto sr = make_rsrc(p.k_scale + row0, (uint32_t)(nrows * 4));
#pragma unroll
        for (int j = 0; j < S::KL; ++j) c.ks[j] = __uint_as_float(buffer_load4(sr, kgrp * 4, j * S::TPK * 4));
    }
#pragma unroll
    for (int j = 0; j < S::VL; ++j) c.v[j] = buffer_load16(vr, voff, j * S::TPV * DV * 2);
    return true;
}

// Online-softmax state of one lane. After the row sums every lane of a key row
// holds the scores of all HG heads; lane kpart (= lane % LPT) keeps heads
// kpart, kpart + LPT, ... (NH of them), so each score is exponentiated once,
// without divergent branches. m and l are the reference maximum (log2 domain)
// and this lane's share of the normaliser of those heads; o holds this lane's
// output columns of every head, summed over the tokens this lane's row group saw.
template <int HG, int NH>
struct LaneState {
    float m[NH], l[NH], o[HG][8];
};

template <int R, int DV, int HG, int KF, int CH>
struct LaneHeads {
    static constexpr int LPT = DecodeShape<R, DV, HG, KF, CH>::LPT;
    static constexpr int NH = (HG + LPT - 1) / LPT;
};

// The reference maximum of a head moves only when a score exceeds it by more
// than kLazy (log2 units), so probabilities stay below 2^kLazy and most chunks
// need no cross-lane maximum at all. Any reference at or above the true
// maximum minus kLazy gives the same softmax (the shift cancels in O / l).
constexpr float kLazy = 8.f;

// Folds one chunk into the lane's state; rows t >= nvalid of the chunk are
// outside the context (their scores become -inf and their values zero, since
// cache memory past the context may hold anything).
template <int R, int DV, int HG, int KF, int CH>
__device__ __forceinline__ void process_chunk(Chunk<R, DV, HG, KF, CH>& c, int nvalid,
                                              LaneState<HG, LaneHeads<R, DV, HG, KF, CH>::NH>& st,
                                              const uint32_t (&qp)[HG][DecodeShape<R, DV, HG, KF, CH>::QW],
                                              const float (&qsum)[HG], float qscale, uint16_t* p16, int lane) {
    using S = DecodeShape<R, DV, HG, KF, CH>;
    constexpr int LPT = S::LPT;
    constexpr int NH = LaneHeads<R, DV, HG, KF, CH>::NH;
    const int kgrp = lane / LPT, kpart = lane % LPT;
    const int vgrp = lane / S::LPV;
    if (nvalid < CH) {  // wave-uniform: only the last chunk of a context
#pragma unroll
        for (int j = 0; j < S::VL; ++j)
            if (j * S::TPV + vgrp >= nvalid) c.v[j] = make_uint4(0, 0, 0, 0);
    }

    // ---- scores (log2 domain) of this lane's key rows, for the lane's own heads
    float sv[S::KL][NH];
#pragma unroll
    for (int j = 0; j < S::KL; ++j) {
        uint32_t kb[S::QW];  // key slice as packed bf16 pairs
        if constexpr (KF == kKeyInt4) {
            // nibble n -> bf16 128 + n (exponent byte 0x43, n in the low mantissa
            // bits), pairs (entry 2m, entry 2m + 1); the excess 136 = 128 + 8 per
            // entry is taken off with the query slice sum below
            const uint32_t w[2] = {c.k[j].x, c.k[j].y};
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const uint32_t lo = w[i] & 0x0f0f0f0fu, hi = (w[i] >> 4) & 0x0f0f0f0fu;
#pragma unroll
                for (int m = 0; m < 4; ++m)
                    kb[4 * i + m] = __builtin_amdgcn_perm(hi, lo, 0x0c040c00u + 0x00010001u * m) | 0x43004300u;
            }
        } else {
            const uint32_t w[4] = {c.k[j].x, c.k[j].y, c.k[j].z, c.k[j].w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if constexpr (KF == kKeyE4M3) {
                    kb[2 * i] = e4m3x2_bf16<false>(w[i]);
                    kb[2 * i + 1] = e4m3x2_bf16<true>(w[i]);
                } else {
                    kb[i] = w[i];
                }
            }
        }
        const bool valid = j * S::TPK + kgrp < nvalid;
        const float sc = KeyRow<KF>::SCALED ? qscale * c.ks[KeyRow<KF>::SCALED ? j : 0] : qscale;
        float acc[HG];
#pragma unroll
        for (int h = 0; h < HG; ++h) {
            float a = 0.f;
#pragma unroll
            for (int i = 0; i < S::QW; ++i) a = dot2_bf16(kb[i], qp[h][i], a);
            if constexpr (KF == kKeyInt4) a = fmaf(-136.f, qsum[h], a);
            acc[h] = group_sum<LPT>(a);
        }
#pragma unroll
        for (int i = 0; i < NH; ++i) {
            float v = acc[i * LPT];
#pragma unroll
            for (int t = 1; t < LPT; ++t)
                if (i * LPT + t < HG) v = kpart == t ? acc[i * LPT + t] : v;
            if (HG % LPT != 0 && kpart + i * LPT >= HG) v = -INFINITY;  // lane without a head here
            sv[j][i] = valid ? v * sc : -INFINITY;
        }
    }

    // ---- the lazy reference maximum: a wave reduction only when some score
    // exceeds its head's reference by more than kLazy (always on the first chunk)
    bool grow = false;
#pragma unroll
    for (int i = 0; i < NH; ++i)
#pragma unroll
        for (int j = 0; j < S::KL; ++j) grow |= sv[j][i] > st.m[i] + kLazy;
    if (__builtin_amdgcn_ballot_w64(grow) != 0) {  // wave-uniform
#pragma unroll
        for (int i = 0; i < NH; ++i) {
            float cm = sv[0][i];
#pragma unroll
            for (int j = 1; j < S::KL; ++j) cm = fmaxf(cm, sv[j][i]);
            cm = strided_max<LPT>(cm);  // over the lanes that own the same heads
            const bool up = cm > st.m[i];
            const float alpha = up ? exp2_fast(st.m[i] - cm) : 1.f;
            st.m[i] = up ? cm : st.m[i];
            st.l[i] *= alpha;
            // every lane holds output columns of every head: take each head's
            // factor from lane t, which owns head i * LPT + t
#pragma unroll
            for (int t = 0; t < LPT; ++t) {
                const int h = i * LPT + t;
                if (h < HG) {
                    const float ah = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(alpha), t));
#pragma unroll
                    for (int e = 0; e < 8; ++e) st.o[h][e] *= ah;
                }
            }
        }
    }

    // ---- probabilities of the lane's heads, rounded to bf16, into the LDS pair
    // table: entry (pair slot, head) holds the tokens of value loads 2q and 2q+1
    // that the same lane will combine
#pragma unroll
    for (int j = 0; j < S::KL; ++j) {
        const int t = j * S::TPK + kgrp;
        const int jv = t / S::TPV, gv = t % S::TPV;
        const int slot = ((jv >> 1) * S::TPV + gv) * HG;
#pragma unroll
        for (int i = 0; i < NH; ++i) {
            const int h = kpart + i * LPT;
            if (HG % LPT == 0 || h < HG) {
                const float pr = exp2_fast(sv[j][i] - st.m[i]);
                const uint32_t pb = pack_bf16(pr, 0.f) & 0xffffu;
                st.l[i] += __uint_as_float(pb << 16);
                p16[(slot + h) * 2 + (jv & 1)] = (uint16_t)pb;
            }
        }
    }
    wave_lds_sync();

    // ---- value rows: token pairs (t1, t2) of loads 2q, 2q+1 against (p1, p2) with dot2
    const uint32_t* p32 = (const uint32_t*)p16;
#pragma unroll
    for (int q = 0; q < S::VL / 2; ++q) {
        uint32_t pp[HG];
#pragma unroll
        for (int h = 0; h < HG; ++h) pp[h] = p32[(q * S::TPV + vgrp) * HG + h];
        const uint32_t a[4] = {c.v[2 * q].x, c.v[2 * q].y, c.v[2 * q].z, c.v[2 * q].w};
        const uint32_t bq[4] = {c.v[2 * q + 1].x, c.v[2 * q + 1].y, c.v[2 * q + 1].z, c.v[2 * q + 1].w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t lo = lo_halves(a[i], bq[i]);  // column 2i of (t1, t2)
            const uint32_t hi = hi_halves(a[i], bq[i]);  // column 2i+1
#pragma unroll
            for (int h = 0; h < HG; ++h) {
                st.o[h][2 * i] = dot2_bf16(lo, pp[h], st.o[h][2 * i]);
                st.o[h][2 * i + 1] = dot2_bf16(hi, pp[h], st.o[h][2 * i + 1]);
            }
        }
    }
    wave_lds_sync();
}

// Two four-wave workgroups per CU where the registers allow it; 4-bit keys with
// eight heads per workgroup (their unpacked query slices are twice as wide), and
// every eight-wave form, take the whole register file of one.
template <int HG, int KF, int NW>
constexpr int decode_min_blocks() { return NW == kDecodeWavesLong && !(KF == kKeyInt4 && HG == 8) ? 2 : 1; }

template <int R, int DV, int HG, int KF, bool PAGED, int NW>
__global__ __launch_bounds__(64 * NW, (decode_min_blocks<HG, KF, NW>())) void decode_split_kernel(
    const DecodeParams p) {
    constexpr int kDecodeWaves = NW;
    constexpr int kDecodeThreads = 64 * NW;
    constexpr int CH = DecodeSchedule<R, DV, HG, KF>::CH;
    constexpr bool PIPE = DecodeSchedule<R, DV, HG, KF>::PIPE;
    using S = DecodeShape<R, DV, HG, KF, CH>;
    constexpr int LPV = S::LPV;
    constexpr int ROWS = 64 / LPV;  // lane row groups of a value load (different tokens, same columns)
    constexpr int LPT = S::LPT;
    constexpr int NH = LaneHeads<R, DV, HG, KF, CH>::NH;

    __shared__ uint32_t p_lds[kDecodeWaves][CH * HG / 2];
    __shared__ float m_lds[kDecodeWaves][HG];
    __shared__ float l_lds[kDecodeWaves][HG];
    __shared__ float o_lds[kDecodeWaves][HG][ROWS][DV];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int split = blockIdx.x;
    const int groups_per_kv = p.G / HG;
    const int g = blockIdx.y / groups_per_kv;
    const int h0 = g * p.G + (blockIdx.y % groups_per_kv) * HG;
    const int b = blockIdx.z;

    // this lane's query slice as packed bf16 pairs (exact; the scale is applied in fp32)
    uint32_t qp[HG][S::QW];
    const int kpart = lane % LPT;
#pragma unroll
    for (int h = 0; h < HG; ++h) {
        const uint4* qrow = (const uint4*)(p.q + ((size_t)b * p.Hq + h0 + h) * R + kpart * S::EPL);
#pragma unroll
        for (int i = 0; i < S::QW / 4; ++i) {
            const uint4 w = qrow[i];
            qp[h][4 * i] = w.x;
            qp[h][4 * i + 1] = w.y;
            qp[h][4 * i + 2] = w.z;
            qp[h][4 * i + 3] = w.w;
        }
    }
    // 4-bit keys: sum of this lane's query slice per head
    float qsum[HG];
#pragma unroll
    for (int h = 0; h < HG; ++h) {
        qsum[h] = 0.f;
        if constexpr (KF == kKeyInt4) {
#pragma unroll
            for (int i = 0; i < S::QW; ++i) qsum[h] += bf16lo(qp[h][i]) + bf16hi(qp[h][i]);
        }
    }

    LaneState<HG, NH> st;
#pragma unroll
    for (int i = 0; i < NH; ++i) {
        st.m[i] = -INFINITY;
        st.l[i] = 0.f;
    }
#pragma unroll
    for (int h = 0; h < HG; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) st.o[h][e] = 0.f;
    bool bad_block = false;
    uint16_t* p16 = (uint16_t*)p_lds[wave];

    // Chunks ts, ts + kStride, ... of this wave: a round is kDecodeWaves chunks,
    // one per wave, and split s takes rounds s, s + n_split, ... With PIPE the
    // next chunk's loads are issued before the current one is processed. For a
    // contiguous cache the first chunk is requested before the context length
    // is read (rows up to max_ctx are readable), so the length's round trip
    // overlaps the stream; paged caches wait for it, because table entries past
    // the context need not be valid.
    using C = Chunk<R, DV, HG, KF, CH>;
    const int kStride = p.n_split * kDecodeWaves * CH;
    int ts = (split * kDecodeWaves + wave) * CH;
    int first_avail = p.max_ctx;
    C ca;
    bool ok_a = true;
    if constexpr (!PAGED) {
        if (ts < first_avail) ok_a = load_chunk<R, DV, HG, KF, CH, PAGED>(ca, p, b, g, ts, first_avail, lane);
        asm volatile("" ::: "memory");  // keep the length's load behind the chunk's loads
    }
    int L = load_uniform(p.ctx_lens + b);
    L = L < 0 ? 0 : (L > p.max_ctx ? p.max_ctx : L);
    const int split_end = L;  // every split walks to the end of the context
    if constexpr (PAGED) {
        first_avail = split_end;
        if (ts < first_avail) ok_a = load_chunk<R, DV, HG, KF, CH, PAGED>(ca, p, b, g, ts, first_avail, lane);
    }
    if (ts < first_avail) {
        if constexpr (PIPE) {
            C cb;
            bool ok_b = true;
            while (true) {
                const bool more_b = ts + kStride < split_end;
                if (more_b) ok_b = load_chunk<R, DV, HG, KF, CH, PAGED>(cb, p, b, g, ts + kStride, split_end, lane);
                if (ts < split_end) {
                    bad_block |= !ok_a;
                    if (ok_a) process_chunk<R, DV, HG, KF, CH>(ca, split_end - ts < CH ? split_end - ts : CH, st, qp,
                                                                qsum, p.qscale, p16, lane);
                }
                if (!more_b) break;
                ts += kStride;
                const bool more_a = ts + kStride < split_end;
                if (more_a) ok_a = load_chunk<R, DV, HG, KF, CH, PAGED>(ca, p, b, g, ts + kStride, split_end, lane);
                bad_block |= !ok_b;
                if (ok_b) process_chunk<R, DV, HG, KF, CH>(cb, split_end - ts < CH ? split_end - ts : CH, st, qp,
                                                            qsum, p.qscale, p16, lane);
                if (!more_a) break;
                ts += kStride;
            }
        } else {
            while (true) {
                if (ts < split_end) {
                    bad_block |= !ok_a;
                    if (ok_a) process_chunk<R, DV, HG, KF, CH>(ca, split_end - ts < CH ? split_end - ts : CH, st, qp,
                                                                qsum, p.qscale, p16, lane);
                }
                ts += kStride;
                if (ts >= split_end) break;
                ok_a = load_chunk<R, DV, HG, KF, CH, PAGED>(ca, p, b, g, ts, split_end, lane);
            }
        }
    }

    // ---- this wave's partial into LDS: the raw output sums of every lane row
    // group (summed over the groups by the merge below), and per head the
    // reference maximum and the normaliser summed over the lanes owning the head
    const bool wave_bad = bad_block;  // wave-uniform
#pragma unroll
    for (int h = 0; h < HG; ++h) {
        float* dst = &o_lds[wave][h][lane / LPV][(lane % LPV) * 8];
        *(float4*)dst = make_float4(st.o[h][0], st.o[h][1], st.o[h][2], st.o[h][3]);
        *(float4*)(dst + 4) = make_float4(st.o[h][4], st.o[h][5], st.o[h][6], st.o[h][7]);
    }
#pragma unroll
    for (int i = 0; i < NH; ++i) {
        const float li = strided_sum<LPT>(st.l[i]);
        const int h = kpart + i * LPT;
        if (lane < LPT && h < HG) {
            m_lds[wave][h] = st.m[i];
            l_lds[wave][h] = wave_bad ? NAN : li;
        }
    }
    __syncthreads();

    // ---- merge the waves (log-sum-exp rule). Each thread owns kOut output
    // columns and reads all of their LDS entries before combining them. With a
    // single split that is the answer: normalise and write the bf16 rows directly.
    constexpr int kOut = (HG * DV + kDecodeThreads - 1) / kDecodeThreads;
    const int ws_row = DV + 2;
    float M[kOut], O[kOut], Lsum[kOut];
    bool bad[kOut];
#pragma unroll
    for (int u = 0; u < kOut; ++u) {
        const int idx = threadIdx.x + u * kDecodeThreads;
        M[u] = -INFINITY;
        O[u] = 0.f;
        Lsum[u] = 0.f;
        bad[u] = false;
        if (idx >= HG * DV) continue;
        const int h = idx / DV, c = idx % DV;
        float mw[kDecodeWaves], lw[kDecodeWaves], ow[kDecodeWaves];
#pragma unroll
        for (int w = 0; w < kDecodeWaves; ++w) {
            mw[w] = m_lds[w][h];
            lw[w] = l_lds[w][h];
            ow[w] = 0.f;
#pragma unroll
            for (int r = 0; r < ROWS; ++r) ow[w] += o_lds[w][h][r][c];
            M[u] = fmaxf(M[u], mw[w]);
        }
#pragma unroll
        for (int w = 0; w < kDecodeWaves; ++w) {
            const float e = mw[w] == -INFINITY ? 0.f : exp2_fast(mw[w] - M[u]);
            O[u] = fmaf(e, ow[w], O[u]);
            Lsum[u] = fmaf(e, lw[w], Lsum[u]);
            bad[u] |= __builtin_isnan(lw[w]);
        }
    }
    if (p.n_split == 1) {
#pragma unroll
        for (int u = 0; u < kOut; ++u) {
            const int idx = threadIdx.x + u * kDecodeThreads;
            if (idx >= HG * DV) continue;
            const int h = idx / DV, c = idx % DV;
            const float out = bad[u] ? NAN : (M[u] == -INFINITY ? 0.f : O[u] / Lsum[u]);
            p.o[((size_t)b * p.Hq + h0 + h) * DV + c] = (uint16_t)(pack_bf16(out, 0.f) & 0xffffu);
        }
        return;
    }
    // Otherwise write this split's partial. Partials are written and read with
    // agent-scope atomic accesses (coherent across the XCDs' separate L2
    // caches without an L2 write-back).
#pragma unroll
    for (int u = 0; u < kOut; ++u) {
        const int idx = threadIdx.x + u * kDecodeThreads;
        if (idx >= HG * DV) continue;
        const int h = idx / DV, c = idx % DV;
        float* dst = p.ws + (((size_t)b * p.Hq + h0 + h) * p.n_split + split) * ws_row;
        store_coherent(dst + c, O[u]);
        if (c == 0) {
            store_coherent(dst + DV, M[u]);
            store_coherent(dst + DV + 1, bad[u] ? NAN : Lsum[u]);
        }
    }

    // ---- the last workgroup of this (sequence, head group) to finish merges the
    // splits with the log-sum-exp rule and writes the bf16 output rows
    __shared__ int is_last;
    wait_stores();  // this thread's partial is visible device-wide
    __syncthreads();
    unsigned* counter = p.counters + (size_t)b * gridDim.y + blockIdx.y;
    if (threadIdx.x == 0)
        is_last = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                  (unsigned)(p.n_split - 1);
    __syncthreads();
    if (!is_last) return;
    // one pass over the splits, up to 8 at a time; all loads of a group, for
    // every column this thread owns, are in flight together; the running-maximum
    // rule of the online softmax combines them
#pragma unroll
    for (int u = 0; u < kOut; ++u) {
        M[u] = -INFINITY;
        O[u] = 0.f;
        Lsum[u] = 0.f;
        bad[u] = false;
    }
    for (int s0 = 0; s0 < p.n_split; s0 += 8) {
        const int cnt = p.n_split - s0 < 8 ? p.n_split - s0 : 8;
        float ms[kOut][8], ls[kOut][8], os[kOut][8];
#pragma unroll
        for (int u = 0; u < kOut; ++u) {
            const int idx = threadIdx.x + u * kDecodeThreads;
            if (idx >= HG * DV) continue;
            const int h = idx / DV, c = idx % DV;
            const float* base = p.ws + ((size_t)b * p.Hq + h0 + h) * p.n_split * ws_row;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                if (i < cnt) {
                    const float* part = base + (size_t)(s0 + i) * ws_row;
                    ms[u][i] = load_coherent(part + DV);
                    ls[u][i] = load_coherent(part + DV + 1);
                    os[u][i] = load_coherent(part + c);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kOut; ++u) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                if (i >= cnt || threadIdx.x + u * kDecodeThreads >= HG * DV) break;
                bad[u] |= __builtin_isnan(ls[u][i]);
                if (ms[u][i] == -INFINITY) continue;
                if (ms[u][i] > M[u]) {
                    const float alpha = exp2_fast(M[u] - ms[u][i]);
                    O[u] *= alpha;
                    Lsum[u] *= alpha;
                    M[u] = ms[u][i];
                }
                const float e = exp2_fast(ms[u][i] - M[u]);
                O[u] = fmaf(e, os[u][i], O[u]);
                Lsum[u] = fmaf(e, ls[u][i], Lsum[u]);
            }
        }
    }
#pragma unroll
    for (int u = 0; u < kOut; ++u) {
        const int idx = threadIdx.x + u * kDecodeThreads;
        if (idx >= HG * DV) continue;
        const int h = idx / DV, c = idx % DV;
        // no visible token -> zeros; a flagged bad block-table entry -> NaN
        const float out = bad[u] ? NAN : (M[u] == -INFINITY ? 0.f : O[u] / Lsum[u]);
        p.o[((size_t)b * p.Hq + h0 + h) * DV + c] = (uint16_t)(pack_bf16(out, 0.f) & 0xffffu);
    }
    if (threadIdx.x == 0) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

#ifndef TK_DECODE_SHORT_UNIT
// ------------------------------------------------------------------ planning

DecodePlan plan_decode(int B, int Hq, int Hkv, int max_ctx, int DV) {
    DecodePlan pl{};
    const int G = Hq / Hkv;
    int hg = 8;
    while (G % hg) hg >>= 1;
    pl.heads_per_group = hg;
    const long pairs = (long)B * Hkv * (G / hg);
    // at least 512 tokens per split (four rounds at 32-token chunks): shorter
    // splits leave each wave too few chunks to pipeline, and the last arriver
    // more partials to merge, than their extra workgroups win back
    const long quanta = (max_ctx + 511) / 512;
    const long target_groups = TK_DECODE_TARGET_GROUPS;  // workgroups to keep 256 CUs streaming
    long n_split = (target_groups + pairs - 1) / pairs;
    if (n_split > quanta) n_split = quanta;
    if (n_split > kMaxSplits) n_split = kMaxSplits;
    if (n_split < 1) n_split = 1;
    long split_quanta = quanta > 0 ? (quanta + n_split - 1) / n_split : 1;
    pl.split_len = (int)(split_quanta * 512);
    pl.n_split = max_ctx > 0 ? (int)((max_ctx + pl.split_len - 1) / pl.split_len) : 1;
    // One arrival counter per (sequence, head group). They are used only when
    // the context is split, which needs fewer than TARGET_GROUPS pairs (fewer
    // than twice that after a launch halves the head group), so one fixed
    // leading region serves every shape: counters never land where another
    // shape's call kept its partials, and a workspace can move between shapes.
    pl.counter_bytes = kCounterRegionBytes;
    pl.ws_bytes = pl.counter_bytes + (size_t)B * Hq * pl.n_split * (DV + 2) * sizeof(float);
    return pl;
}

// ------------------------------------------------------------------ fixed scratch

// Callers that cannot allocate (graph capture, tight serving loops) use this
// array instead of a workspace of their own. Host code never passes its name:
// it looks up the device address once per device and uses that.
static __device__ __align__(256) unsigned char scratch[kDecodeScratchBytes];
static_assert(kCounterRegionBytes <= kDecodeScratchBytes, "the counters fit the scratch");

__global__ void zero_words_kernel(unsigned* p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0u;
}

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];  // device address of each device's copy, once looked up
}  // namespace

tk_status decode_scratch(hipStream_t stream, void** ptr) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return TK_ERR_HIP;
    int sdev = -1;
    if (hipStreamGetDevice(stream, &sdev) != hipSuccess) return TK_ERR_HIP;
    if (sdev != dev) return TK_ERR_INVALID_ARG;  // the scratch used is the current device's
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* addr = nullptr;
        if (hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch)) != hipSuccess || !addr) return TK_ERR_HIP;
        // the arrival counters must start at zero; completed calls leave them zero
        const int words = (int)(kCounterRegionBytes / sizeof(unsigned));
        hipLaunchKernelGGL(zero_words_kernel, dim3((words + 255) / 256), dim3(256), 0, stream, (unsigned*)addr,
                           words);
        if (hipGetLastError() != hipSuccess) return TK_ERR_HIP;
        g_scratch[dev] = addr;
    }
    *ptr = g_scratch[dev];
    return TK_OK;
}

#endif  // TK_DECODE_SHORT_UNIT

// ------------------------------------------------------------------ dispatch
//
// The dispatch chain is instantiated twice: for four-wave workgroups in this
// file, and for eight-wave ones in decode_short.hip, which includes this file
// with TK_DECODE_SHORT_UNIT defined (the two sets then compile in parallel).

// Eight-wave launches (decode_short.hip).
tk_status launch_decode_short(const DecodeParams& p, int R, int DV, int HG, int key_format, bool paged,
                              hipStream_t st);

// Whether a layout has an eight-wave form: not 4-bit keys with eight heads per
// workgroup, which need the whole register file of a SIMD for one wave.
template <int HG, int KF>
constexpr bool has_short_form() { return !(KF == kKeyInt4 && HG == 8); }

// Four-wave workgroups, unless they would give each wave at most kShortRounds
// chunks of its split (small batches at short contexts): then eight. The choice
// depends only on the shapes, so a shape's output stays bitwise reproducible.
template <int NW, int R, int DV, int HG, int KF>
static bool use_short(const DecodeParams& p) {
    if constexpr (NW != kDecodeWavesLong || !has_short_form<HG, KF>()) {
        return false;
    } else {
        constexpr int CH = DecodeSchedule<R, DV, HG, KF>::CH;
        const long rounds = ((long)p.max_ctx + kDecodeWavesLong * CH - 1) / (kDecodeWavesLong * CH);
        return (rounds + p.n_split - 1) / p.n_split <= kShortRounds;
    }
}

template <int NW, int R, int DV, int HG, int KF, bool PAGED>
static hipError_t run(const DecodeParams& p, hipStream_t st) {
    if constexpr (NW == kDecodeWavesShort && !has_short_form<HG, KF>()) {
        return hipErrorInvalidValue;  // never chosen (use_short), and not built
    } else {
        if (use_short<NW, R, DV, HG, KF>(p)) {
            const tk_status s = launch_decode_short(p, R, DV, HG, KF, PAGED, st);
            return s == TK_OK ? hipSuccess : (s == TK_ERR_UNSUPPORTED ? hipErrorInvalidValue : hipErrorLaunchFailure);
        }
        const dim3 grid(p.n_split, p.Hkv * (p.G / HG), p.B);
        hipLaunchKernelGGL((decode_split_kernel<R, DV, HG, KF, PAGED, NW>), grid, dim3(64 * NW), 0, st, p);
        return hipGetLastError();
    }
}

template <int NW, int R, int DV, int HG, int KF>
static hipError_t by_paging(const DecodeParams& p, bool paged, hipStream_t st) {
    return paged ? run<NW, R, DV, HG, KF, true>(p, st) : run<NW, R, DV, HG, KF, false>(p, st);
}

template <int NW, int R, int DV, int HG>
static hipError_t by_layout(const DecodeParams& p, int kf, bool paged, hipStream_t st) {
    switch (kf) {
        case kKeyBF16: return by_paging<NW, R, DV, HG, kKeyBF16>(p, paged, st);
        case kKeyE4M3: return by_paging<NW, R, DV, HG, kKeyE4M3>(p, paged, st);
        case kKeyInt4: return by_paging<NW, R, DV, HG, kKeyInt4>(p, paged, st);
        default: return hipErrorInvalidValue;
    }
}

template <int NW, int R, int DV>
static hipError_t by_group(const DecodeParams& p, int HG, int kf, bool paged, hipStream_t st) {
    switch (HG) {
        case 1: return by_layout<NW, R, DV, 1>(p, kf, paged, st);
        case 2: return by_layout<NW, R, DV, 2>(p, kf, paged, st);
        case 4: return by_layout<NW, R, DV, 4>(p, kf, paged, st);
        case 8:
            // eight heads per workgroup only for r < 64; wider keys take four (their
            // eight-head form would not fit the register budget)
            if constexpr (R < 64) return by_layout<NW, R, DV, 8>(p, kf, paged, st);
            return hipErrorInvalidValue;
        default: return hipErrorInvalidValue;
    }
}

template <int NW, int R>
static hipError_t by_dv(const DecodeParams& p, int DV, int HG, int kf, bool paged, hipStream_t st) {
    if (DV == 64) return by_group<NW, R, 64>(p, HG, kf, paged, st);
    if (DV == 128) return by_group<NW, R, 128>(p, HG, kf, paged, st);
    return hipErrorInvalidValue;
}

template <int NW>
static tk_status launch_waves(const DecodeParams& p, int R, int DV, int HG, int key_format, bool paged,
                              hipStream_t st) {
    hipError_t e;
    switch (R) {
        case 16: e = by_dv<NW, 16>(p, DV, HG, key_format, paged, st); break;
        case 32: e = by_dv<NW, 32>(p, DV, HG, key_format, paged, st); break;
        case 64: e = by_dv<NW, 64>(p, DV, HG, key_format, paged, st); break;
        case 128: e = by_dv<NW, 128>(p, DV, HG, key_format, paged, st); break;
        default: return TK_ERR_UNSUPPORTED;
    }
    if (e == hipErrorInvalidValue) return TK_ERR_UNSUPPORTED;
    return e == hipSuccess ? TK_OK : TK_ERR_HIP;
}

#ifdef TK_DECODE_SHORT_UNIT
tk_status launch_decode_short(const DecodeParams& p, int R, int DV, int HG, int key_format, bool paged,
                              hipStream_t st) {
    return launch_waves<kDecodeWavesShort>(p, R, DV, HG, key_format, paged, st);
}
#else
tk_status launch_decode(const DecodeParams& p, int R, int DV, int HG, int key_format, bool paged, hipStream_t st) {
    return launch_waves<kDecodeWavesLong>(p, R, DV, HG, key_format, paged, st);
}
#endif

}  // namespace tk
