// Thin-key decode attention for gfx950: split-K over the cached context.
//
// One decode step reads every cached key row (r entries) and value row (d_v
// entries) once; that stream dominates the step's memory traffic, which is why
// decode is bandwidth-bound (Sec. 4.2, Eq. 10) and why thin keys cut its cost
// by (r + d_v) / (2 d_head) (Eq. 8-9). The kernels here are built around that:
//
//  * Grouped-query packing: a workgroup serves all HG query heads that share a
//    KV head, so each K/V byte crosses HBM once for HG heads.
//  * Each wave streams 64-token chunks with 16-byte loads per lane, all of a
//    chunk's K and V loads issued before any arithmetic: key rows tile the lanes
//    (LPT lanes per row, one 16-byte slice each), value rows likewise.
//  * Scores: per-lane partial dot products over the lane's slice of r, reduced
//    across the LPT lanes of a row with DPP. The softmax scale and log2(e) are
//    folded into the fp32 query once, so the softmax uses exp2 directly; for
//    fp8 keys the per-(token, head) scale multiplies the reduced dot product.
//  * Online softmax per head with a wave-wide running maximum; probabilities go
//    through a small per-wave LDS table to the lanes that own the value columns.
//  * The 4 waves of a workgroup merge their (max, sum, output) triples in LDS
//    and write one partial per (sequence, head, split). The last workgroup of a
//    (sequence, head group) to finish - found with an agent-scope counter in the
//    workspace, which it resets to zero - merges the splits with the log-sum-exp
//    rule and writes bf16, so one call is one kernel launch.
#include "tk_device.hpp"
#include "tk_internal.hpp"

#include <math.h>

namespace tk {

constexpr int kDecodeThreads = 256;
constexpr int kDecodeWaves = kDecodeThreads / 64;
constexpr int kChunk = 64;  // tokens per wave iteration
constexpr int kMaxSplits = 256;

// Agent-scope relaxed atomic accesses (sc1 on gfx950): coherent across XCDs.
__device__ __forceinline__ void store_coherent(float* p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_coherent(const float* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Wait until this thread's outstanding global stores have completed.
__device__ __forceinline__ void wait_stores() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

template <int R, int DV, int HG, bool FP8, bool PAGED>
__global__ __launch_bounds__(kDecodeThreads, 2) void decode_split_kernel(const DecodeParams p) {
    constexpr int KB = FP8 ? 1 : 2;        // bytes per key element
    constexpr int ROWB = R * KB;           // bytes per key row
    constexpr int LPT = ROWB / 16;         // lanes per key row
    constexpr int EPL = 16 / KB;           // key elements per lane slice
    constexpr int TPK = 64 / LPT;          // key rows per wave-wide load
    constexpr int KL = LPT;                // key loads per chunk
    constexpr int LPV = DV * 2 / 16;       // lanes per value row
    constexpr int TPV = 64 / LPV;          // value rows per wave-wide load
    constexpr int VL = LPV;                // value loads per chunk
    static_assert(LPT >= 1 && LPT <= 16 && LPV >= 8 && LPV <= 16, "unsupported shape");

    __shared__ float p_lds[kDecodeWaves][kChunk * HG];
    __shared__ float m_lds[kDecodeWaves][HG];
    __shared__ float l_lds[kDecodeWaves][HG];
    __shared__ float o_lds[kDecodeWaves][HG][DV];

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int split = blockIdx.x;
    const int groups_per_kv = p.G / HG;
    const int g = blockIdx.y / groups_per_kv;
    const int h0 = g * p.G + (blockIdx.y % groups_per_kv) * HG;
    const int b = blockIdx.z;

    int L = p.ctx_lens[b];
    L = L < 0 ? 0 : (L > p.max_ctx ? p.max_ctx : L);
    const int split_begin = split * p.split_len;
    int split_end = split_begin + p.split_len;
    split_end = split_end < L ? split_end : L;

    // query slice of this lane, pre-multiplied by scale * log2(e)
    const int kpart = lane % LPT;
    float qf[HG][EPL];
#pragma unroll
    for (int h = 0; h < HG; ++h) {
        const uint16_t* qrow = p.q + ((size_t)b * p.Hq + h0 + h) * R + kpart * EPL;
#pragma unroll
        for (int e = 0; e < EPL; ++e) qf[h][e] = __uint_as_float((uint32_t)qrow[e] << 16) * p.qscale;
    }

    float m[HG], l[HG], o[HG][8];
#pragma unroll
    for (int h = 0; h < HG; ++h) {
        m[h] = -INFINITY;
        l[h] = 0.f;
#pragma unroll
        for (int c = 0; c < 8; ++c) o[h][c] = 0.f;
    }
    bool bad_block = false;

    const int vpart = lane % LPV;
    float* pw = p_lds[wave];

    for (int ts = split_begin + wave * kChunk; ts < split_end; ts += kDecodeWaves * kChunk) {
        const int nvalid = split_end - ts < kChunk ? split_end - ts : kChunk;
        const uint8_t* kbase;
        const uint16_t* vbase;
        const float* sbase = nullptr;
        if constexpr (PAGED) {
            int blk = p.block_table[(size_t)b * p.mb + (ts >> p.bs_log2)];
            blk = __builtin_amdgcn_readfirstlane(blk);
            if (blk < 0 || blk >= p.num_blocks) {  // never dereference a bad entry
                bad_block = true;
                continue;
            }
            const size_t row0 = (((size_t)blk * p.Hkv + g) << p.bs_log2) + (ts & ((1 << p.bs_log2) - 1));
            kbase = p.k + row0 * ROWB;
            vbase = p.v + row0 * DV;
            if constexpr (FP8) sbase = p.k_scale + row0;
        } else {
            const size_t row0 = ((size_t)b * p.Hkv + g) * p.max_ctx + ts;
            kbase = p.k + row0 * ROWB;
            vbase = p.v + row0 * DV;
            if constexpr (FP8) sbase = p.k_scale + row0;
        }

        // ---- issue every load of the chunk
        uint4 kr[KL];
        float ks[KL];
#pragma unroll
        for (int j = 0; j < KL; ++j) {
            const int t = j * TPK + lane / LPT;
            kr[j] = t < nvalid ? *(const uint4*)(kbase + (size_t)t * ROWB + kpart * 16) : make_uint4(0, 0, 0, 0);
            if constexpr (FP8) ks[j] = t < nvalid ? sbase[t] : 0.f;
        }
        uint4 vr[VL];
#pragma unroll
        for (int j = 0; j < VL; ++j) {
            const int t = j * TPV + lane / LPV;
            vr[j] = t < nvalid ? *(const uint4*)(vbase + (size_t)t * DV + vpart * 8) : make_uint4(0, 0, 0, 0);
        }

        // ---- scores (log2 domain) for this lane's key rows, all HG heads
        float s[KL][HG];
#pragma unroll
        for (int j = 0; j < KL; ++j) {
            float kf[EPL];
            const uint32_t w[4] = {kr[j].x, kr[j].y, kr[j].z, kr[j].w};
            if constexpr (FP8) {
#pragma unroll
                for (int i = 0; i < 4; ++i) e4m3x4(w[i], kf[4 * i], kf[4 * i + 1], kf[4 * i + 2], kf[4 * i + 3]);
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    kf[2 * i] = bf16lo(w[i]);
                    kf[2 * i + 1] = bf16hi(w[i]);
                }
            }
            const bool valid = j * TPK + lane / LPT < nvalid;
#pragma unroll
            for (int h = 0; h < HG; ++h) {
                float acc = 0.f;
#pragma unroll
                for (int e = 0; e < EPL; ++e) acc = fmaf(qf[h][e], kf[e], acc);
                acc = group_sum<LPT>(acc);
                if constexpr (FP8) acc *= ks[j];
                s[j][h] = valid ? acc : -INFINITY;
            }
        }

        // ---- online softmax: chunk maximum per head, rescale the running state
#pragma unroll
        for (int h = 0; h < HG; ++h) {
            float cm = s[0][h];
#pragma unroll
            for (int j = 1; j < KL; ++j) cm = fmaxf(cm, s[j][h]);
            cm = strided_max<LPT>(cm);
            const float mn = fmaxf(m[h], cm);
            const float alpha = exp2_fast(m[h] - mn);
            m[h] = mn;
            l[h] *= alpha;
#pragma unroll
            for (int c = 0; c < 8; ++c) o[h][c] *= alpha;
        }

        // ---- probabilities: lane (row slice kpart) computes heads h == kpart (mod LPT)
#pragma unroll
        for (int j = 0; j < KL; ++j) {
            const int t = j * TPK + lane / LPT;
#pragma unroll
            for (int h = 0; h < HG; ++h) {
                if (h % LPT == kpart) {
                    const float pr = exp2_fast(s[j][h] - m[h]);
                    l[h] += pr;
                    pw[t * HG + h] = pr;
                }
            }
        }
        wave_lds_sync();

        // ---- value rows weighted by the probabilities of their token
#pragma unroll
        for (int j = 0; j < VL; ++j) {
            const int t = j * TPV + lane / LPV;
            float pr[HG];
#pragma unroll
            for (int h = 0; h < HG; ++h) pr[h] = pw[t * HG + h];
            const uint32_t w[4] = {vr[j].x, vr[j].y, vr[j].z, vr[j].w};
            float vf[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                vf[2 * i] = bf16lo(w[i]);
                vf[2 * i + 1] = bf16hi(w[i]);
            }
#pragma unroll
            for (int h = 0; h < HG; ++h)
#pragma unroll
                for (int c = 0; c < 8; ++c) o[h][c] = fmaf(pr[h], vf[c], o[h][c]);
        }
        wave_lds_sync();
    }

    // ---- wave totals: sums over the lanes that saw different rows
#pragma unroll
    for (int h = 0; h < HG; ++h) {
        l[h] = strided_sum<1>(l[h]);
#pragma unroll
        for (int c = 0; c < 8; ++c) o[h][c] = strided_sum<LPV>(o[h][c]);
    }
    const bool wave_bad = __any(bad_block);
    if (lane < LPV) {
#pragma unroll
        for (int h = 0; h < HG; ++h)
#pragma unroll
            for (int c = 0; c < 8; ++c) o_lds[wave][h][lane * 8 + c] = o[h][c];
    }
    if (lane == 0) {
#pragma unroll
        for (int h = 0; h < HG; ++h) {
            m_lds[wave][h] = m[h];
            l_lds[wave][h] = wave_bad ? NAN : l[h];
        }
    }
    __syncthreads();

    // ---- merge the 4 waves and write this split's partial per head. Partials are
    // written and read with agent-scope atomic accesses (coherent across the
    // XCDs' separate L2 caches without an L2 write-back).
    const int ws_row = DV + 2;
    for (int idx = threadIdx.x; idx < HG * DV; idx += kDecodeThreads) {
        const int h = idx / DV, c = idx % DV;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kDecodeWaves; ++w) M = fmaxf(M, m_lds[w][h]);
        float O = 0.f, Lsum = 0.f;
#pragma unroll
        for (int w = 0; w < kDecodeWaves; ++w) {
            const float mw = m_lds[w][h];
            const float e = mw == -INFINITY ? 0.f : exp2_fast(mw - M);
            O = fmaf(e, o_lds[w][h][c], O);
            Lsum = fmaf(e, l_lds[w][h], Lsum);
            if (__builtin_isnan(l_lds[w][h])) Lsum = NAN;
        }
        float* dst = p.ws + (((size_t)b * p.Hq + h0 + h) * p.n_split + split) * ws_row;
        store_coherent(dst + c, O);
        if (c == 0) {
            store_coherent(dst + DV, M);
            store_coherent(dst + DV + 1, Lsum);
        }
    }

    // ---- the last workgroup of this (sequence, head group) to finish merges the
    // splits with the log-sum-exp rule and writes the bf16 output rows
    __shared__ int is_last;
    __shared__ float w_lds[HG][kMaxSplits];   // per-split weights exp2(m_s - M)
    __shared__ float inv_l_lds[HG];
    wait_stores();  // this thread's partial is visible device-wide
    __syncthreads();
    unsigned* counter = p.counters + (size_t)b * gridDim.y + blockIdx.y;
    if (threadIdx.x == 0)
        is_last = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                  (unsigned)(p.n_split - 1);
    __syncthreads();
    if (!is_last) return;
    for (int h = wave; h < HG; h += kDecodeWaves) {  // a wave per head: maximum, weights, normaliser
        const float* base = p.ws + ((size_t)b * p.Hq + h0 + h) * p.n_split * ws_row;
        float M = -INFINITY;
        for (int sp = lane; sp < p.n_split; sp += 64) M = fmaxf(M, load_coherent(base + (size_t)sp * ws_row + DV));
        M = group_max<64>(M);
        float Lsum = 0.f;
        bool bad = false;
        for (int sp = lane; sp < p.n_split; sp += 64) {
            const float ms = load_coherent(base + (size_t)sp * ws_row + DV);
            const float ls = load_coherent(base + (size_t)sp * ws_row + DV + 1);
            const float e = ms == -INFINITY ? 0.f : exp2_fast(ms - M);
            w_lds[h][sp] = e;
            Lsum = fmaf(e, ls, Lsum);
            bad |= __builtin_isnan(ls);
        }
        Lsum = group_sum<64>(Lsum);
        // no visible token -> zeros; a flagged bad block-table entry -> NaN
        if (lane == 0) inv_l_lds[h] = __any(bad) ? NAN : (M == -INFINITY ? 0.f : 1.f / Lsum);
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < HG * DV; idx += kDecodeThreads) {
        const int h = idx / DV, c = idx % DV;
        const float* base = p.ws + ((size_t)b * p.Hq + h0 + h) * p.n_split * ws_row + c;
        float O = 0.f;
        for (int sp = 0; sp < p.n_split; ++sp) O = fmaf(w_lds[h][sp], load_coherent(base + (size_t)sp * ws_row), O);
        const float il = inv_l_lds[h];
        const float out = __builtin_isnan(il) ? NAN : O * il;
        p.o[((size_t)b * p.Hq + h0 + h) * DV + c] = (uint16_t)(pack_bf16(out, 0.f) & 0xffffu);
    }
    if (threadIdx.x == 0) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------------ planning

DecodePlan plan_decode(int B, int Hq, int Hkv, int max_ctx, int DV) {
    DecodePlan pl{};
    const int G = Hq / Hkv;
    int hg = 8;
    while (G % hg) hg >>= 1;
    pl.heads_per_group = hg;
    const long pairs = (long)B * Hkv * (G / hg);
    const long quanta = (max_ctx + 255) / 256;  // 256 tokens = one chunk per wave
    const long target_groups = 1024;             // workgroups to keep 256 CUs streaming
    long n_split = (target_groups + pairs - 1) / pairs;
    if (n_split > quanta) n_split = quanta;
    if (n_split > kMaxSplits) n_split = kMaxSplits;
    if (n_split < 1) n_split = 1;
    long split_quanta = quanta > 0 ? (quanta + n_split - 1) / n_split : 1;
    pl.split_len = (int)(split_quanta * 256);
    pl.n_split = max_ctx > 0 ? (int)((max_ctx + pl.split_len - 1) / pl.split_len) : 1;
    pl.counter_bytes = ((size_t)B * (Hq / hg) * sizeof(unsigned) + 255) / 256 * 256;
    pl.ws_bytes = pl.counter_bytes + (size_t)B * Hq * pl.n_split * (DV + 2) * sizeof(float);
    return pl;
}

// ------------------------------------------------------------------ dispatch

template <int R, int DV, int HG, bool FP8, bool PAGED>
static hipError_t run(const DecodeParams& p, hipStream_t st) {
    dim3 grid(p.n_split, p.Hkv * (p.G / HG), p.B);
    hipLaunchKernelGGL((decode_split_kernel<R, DV, HG, FP8, PAGED>), grid, dim3(kDecodeThreads), 0, st, p);
    return hipGetLastError();
}

template <int R, int DV, int HG>
static hipError_t by_layout(const DecodeParams& p, bool fp8, bool paged, hipStream_t st) {
    if (fp8) return paged ? run<R, DV, HG, true, true>(p, st) : run<R, DV, HG, true, false>(p, st);
    return paged ? run<R, DV, HG, false, true>(p, st) : run<R, DV, HG, false, false>(p, st);
}

template <int R, int DV>
static hipError_t by_group(const DecodeParams& p, int HG, bool fp8, bool paged, hipStream_t st) {
    switch (HG) {
        case 1: return by_layout<R, DV, 1>(p, fp8, paged, st);
        case 2: return by_layout<R, DV, 2>(p, fp8, paged, st);
        case 4: return by_layout<R, DV, 4>(p, fp8, paged, st);
        case 8: return by_layout<R, DV, 8>(p, fp8, paged, st);
        default: return hipErrorInvalidValue;
    }
}

template <int R>
static hipError_t by_dv(const DecodeParams& p, int DV, int HG, bool fp8, bool paged, hipStream_t st) {
    if (DV == 64) return by_group<R, 64>(p, HG, fp8, paged, st);
    if (DV == 128) return by_group<R, 128>(p, HG, fp8, paged, st);
    return hipErrorInvalidValue;
}

tk_status launch_decode(const DecodeParams& p, int R, int DV, int HG, bool fp8, bool paged, hipStream_t st) {
    hipError_t e;
    switch (R) {
        case 16: e = by_dv<16>(p, DV, HG, fp8, paged, st); break;
        case 32: e = by_dv<32>(p, DV, HG, fp8, paged, st); break;
        case 64: e = by_dv<64>(p, DV, HG, fp8, paged, st); break;
        case 128: e = by_dv<128>(p, DV, HG, fp8, paged, st); break;
        default: return TK_ERR_UNSUPPORTED;
    }
    if (e == hipErrorInvalidValue) return TK_ERR_UNSUPPORTED;
    return e == hipSuccess ? TK_OK : TK_ERR_HIP;
}

}  // namespace tk
