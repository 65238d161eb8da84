// Thin-key prefill attention for gfx950 with fp32 inputs and fp32 matrix cores
// (v_mfma_f32_16x16x4_f32), for callers that need fp32 accuracy (bf16 operands
// would not hold a 1e-4 error bound).
//
// Work decomposition. The fp32 matrix instructions are slow (64 FLOPs per cycle
// per SIMD), so a causal prefill is bound by its longest query block, whose
// whole key prefix runs on one CU. A workgroup therefore holds ONE block of 16
// query rows of one head (half the matrix work of a 32-row block per key), and
// its 4 waves split that block's key tiles among themselves (wave w takes tiles
// w, w + 4, ...), each wave with its own tile in LDS and its own online-softmax
// state; the 4 partial results are merged in LDS with the log-sum-exp rule at
// the end. Workgroups are ranked by prefix length across heads and sequences,
// longest first, so the round-robin dispatch deals every XCD the same mix; every
// other round of 256 workgroups (one per CU) takes its ranks in reverse, so a CU
// that received one of the longest blocks in one round receives one of the
// shorter blocks of the next.
//
// Inside a wave: transposed scores S^T = K Q^T per 16-key block, so lane (g, n)
// of lane group g = lane / 16 serves query n = lane % 16, and O^T = V^T P^T.
// Each instruction contracts 4 indices, one per lane group, so:
//  * the score product walks r in R/4 steps, lane group g covering dims
//    [g R/4, (g+1) R/4) (contiguous in the K row, read 16 bytes at a time);
//  * the value product takes, in step i of a key block, keys 4 g + i: the keys
//    whose scores lane group g already holds in accumulator register i, so P^T
//    is used in place with no repacking. V stays in its natural [keys][d_v]
//    layout in LDS (rows padded by 16 bytes, so the four lane groups' rows fall
//    on disjoint banks); a lane reads its four keys of one column with two
//    paired 4-byte reads. A transposed copy would give one 16-byte read instead,
//    but the transpose has to be done in registers, and the fp32 matrix
//    instructions do not overlap VALU work, so those moves cost issue time.
// Row maxima and sums reduce over the four lane groups of a query (lane
// n, n + 16, n + 32, n + 48). A wave loads its next tile into registers while
// it computes the current one; the loads are waited for only when that tile is
// stored to LDS at the top of the next step.
#include "tk_device.hpp"
#include "tk_internal.hpp"

#include <math.h>

namespace tk {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kRows = 16;  // query rows per workgroup

// Keys per tile: 32 (two 16-key blocks). A wave's tile then costs 32 (R + DV) / 64
// floats of prefetch registers per lane, and at the GPT-2 shape (r 16, d_v 64)
// the workgroup's four tiles take 42 KB of LDS, so three workgroups share a CU
// and each SIMD interleaves three waves: while one waits on its dependent
// score -> softmax -> value chain, another issues matrix products (with 64-key
// tiles only one workgroup fits and that chain leaves the matrix core idle for
// about 40 % of a tile).
template <int R, int DV>
struct alignas(16) WaveTile {
    static constexpr int BN = 32;
    static constexpr int KB = BN / 32;  // 32-key blocks per tile
    static constexpr int KS = R;        // floats per K row in LDS (16-byte chunks swizzled by kpos)
    static constexpr int VS = DV + 4;   // floats per V row in LDS (16-byte pad)
    float k[BN * KS];
    float v[BN * VS];
};

// One tile of one wave in registers: 16-byte chunks of K rows and of V rows.
template <int R, int DV>
struct WaveRegs {
    static constexpr int BN = WaveTile<R, DV>::BN;
    static constexpr int KCH = BN * R / 4;
    static constexpr int VCH = BN * DV / 4;
    static_assert(KCH % 64 == 0 && VCH % 64 == 0, "tile does not divide over the lanes");
    static constexpr int KL = KCH / 64;
    static constexpr int VL = VCH / 64;
    float4 k[KL];
    float4 v[VL];
};

// Raw buffer descriptor over `bytes` bytes at `base`: loads past the end return zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const float* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), 0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ float4 load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    typedef float f32x4v __attribute__((ext_vector_type(4)));
    const f32x4v v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
    return make_float4(v[0], v[1], v[2], v[3]);
}

// The tile of keys base .. base + 31, through descriptors that cover just the
// tile's keys below Sk: keys at or past Sk (a ragged last tile) load as zeros by
// the range check, with no per-lane test, and their scores are masked. One load
// path keeps the prefetched registers in place across the loop (two paths
// merged at the loop head made the compiler copy them, and wait for the loads
// to land, right after issuing them).
template <int R, int DV>
__device__ __forceinline__ void load_tile(WaveRegs<R, DV>& t, const float* kg, const float* vg, int base, int Sk,
                                          int lane) {
    using W = WaveRegs<R, DV>;
    constexpr int KC = R / 4, VC = DV / 4;  // 16-byte chunks per K row and per V row
    const uint32_t rows = (uint32_t)(Sk - base < W::BN ? Sk - base : W::BN);
    const auto kr = tile_rsrc(kg + (size_t)base * R, rows * R * 4);
    const auto vr = tile_rsrc(vg + (size_t)base * DV, rows * DV * 4);
#pragma unroll
    for (int i = 0; i < W::KL; ++i) {
        const int c = lane + 64 * i;
        t.k[i] = load16(kr, (uint32_t)(((c / KC) * R + (c % KC) * 4) * 4));
    }
#pragma unroll
    for (int i = 0; i < W::VL; ++i) {
        const int c = lane + 64 * i;
        t.v[i] = load16(vr, (uint32_t)(((c / VC) * DV + (c % VC) * 4) * 4));
    }
}

// Position of 16-byte chunk c of K row r in LDS: rows are R floats, so 256 / (4 R)
// of them share one 256-byte line of the 64 banks (at least one); rotating the
// chunk by the row's line index makes the 16 rows a quarter-wave reads at one
// chunk fall on 16 different 16-byte bank groups, and the stores of whole rows
// stay contiguous per line.
template <int R>
__device__ __forceinline__ int kpos(int r, int c) {
    constexpr int RPL = (64 / R) > 0 ? 64 / R : 1;  // rows per 256-byte line
    constexpr int M = (R / 4 < 16 ? R / 4 : 16) - 1;
    return c ^ ((r / RPL) & M);
}

template <int R, int DV>
__device__ __forceinline__ void store_tile(const WaveRegs<R, DV>& t, WaveTile<R, DV>& tile, int lane) {
    using W = WaveRegs<R, DV>;
    using T = WaveTile<R, DV>;
    constexpr int KC = R / 4, VC = DV / 4;
#pragma unroll
    for (int i = 0; i < W::KL; ++i) {
        const int c = lane + 64 * i;
        *(float4*)(tile.k + (c / KC) * T::KS + kpos<R>(c / KC, c % KC) * 4) = t.k[i];
    }
#pragma unroll
    for (int i = 0; i < W::VL; ++i) {
        const int c = lane + 64 * i;
        *(float4*)(tile.v + (c / VC) * T::VS + (c % VC) * 4) = t.v[i];
    }
}

// LDS of the workgroup: the waves' tiles while streaming, then the waves'
// partial outputs (O^T rows padded to 33 floats), maxima and row sums.
template <int R, int DV>
struct alignas(16) MergeLds {
    float o[kWaves][DV][kRows + 1];
    float m[kWaves][kRows];
    float l[kWaves][kRows];
};
template <int R, int DV>
union alignas(16) Smem {
    WaveTile<R, DV> tile[kWaves];
    MergeLds<R, DV> merge;
};

}  // namespace

template <int R, int DV>
__global__ __launch_bounds__(kThreads, 1) void prefill_f32_kernel(const PrefillParams p) {
    using T = WaveTile<R, DV>;
    constexpr int RS = R / 4;     // score-product steps: lane group g covers dims [g RS, (g + 1) RS)
    constexpr int DBLK = DV / 16;  // 16-row blocks of O^T
    constexpr int BN = T::BN, KS = T::KS, VS = T::VS;
    static_assert(BN == 32, "a tile is two 16-key blocks");
    __shared__ Smem<R, DV> sm;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = lane >> 4, n = lane & 15;  // lane group, and the query (B column) the lane serves

    // workgroup -> (query block, head, sequence): ranked by causal prefix length,
    // longest first, with the heads and sequences of one rank adjacent, so that the
    // round-robin dispatch over the XCDs deals every XCD the same mix of long and
    // short blocks; odd rounds of 256 workgroups take their positions in reverse
    const int nqb = (p.Sq + kRows - 1) / kRows;
    const unsigned round = blockIdx.x / 256u, first = round * 256u;
    const unsigned in_round = (gridDim.x - first < 256u ? gridDim.x - first : 256u);
    const unsigned pos = (round & 1u) ? first + in_round - 1u - (blockIdx.x - first) : blockIdx.x;
    const int rank = (int)(pos / ((unsigned)p.Hq * p.B));
    const int hb = (int)(pos % ((unsigned)p.Hq * p.B));
    const int qb = p.causal ? nqb - 1 - rank : rank;
    const int h = hb % p.Hq;
    const int g = h / p.G;
    const int b = hb / p.Hq;
    const int q0 = qb * kRows;
    const int off = p.Sk - p.Sq;  // bottom-right causal alignment

    const float* qg = (const float*)p.q + ((size_t)b * p.Hq + h) * p.Sq * R;
    const float* kg = (const float*)p.k + ((size_t)b * p.Hkv + g) * p.Sk * R;
    const float* vg = (const float*)p.v + ((size_t)b * p.Hkv + g) * p.Sk * DV;
    float* og = (float*)p.o + ((size_t)b * p.Hq + h) * p.Sq * DV;

    const int qrow = q0 + n;
    float qreg[RS];
#pragma unroll
    for (int s4 = 0; s4 < RS; s4 += 4) {
        const float4 w = qrow < p.Sq ? *(const float4*)(qg + (size_t)qrow * R + grp * RS + s4) : make_float4(0, 0, 0, 0);
        qreg[s4] = w.x;
        qreg[s4 + 1] = w.y;
        qreg[s4 + 2] = w.z;
        qreg[s4 + 3] = w.w;
    }

    int key_end = p.Sk;
    if (p.causal) {
        const int last = q0 + kRows + off;  // one past the last key the block's last row sees
        key_end = last < key_end ? last : key_end;
    }
    const int ntiles = (key_end + BN - 1) / BN;

    f32x4 o[DBLK];
#pragma unroll
    for (int d = 0; d < DBLK; ++d) o[d] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_ref = -INFINITY;  // this query's reference maximum (log2 domain), the same in its 4 lanes
    float lsum = 0.f;         // this lane's share of the query's row sum
    const float c = p.qscale;

    T& tile = sm.tile[wave];
    WaveRegs<R, DV> regs;
    int t = wave;
    if (t < ntiles) load_tile<R, DV>(regs, kg, vg, t * BN, p.Sk, lane);
    for (; t < ntiles; t += kWaves) {
        const int base = t * BN;
        store_tile<R, DV>(regs, tile, lane);
        wave_lds_sync();
        if (t + kWaves < ntiles) load_tile<R, DV>(regs, kg, vg, base + kWaves * BN, p.Sk, lane);

        // S^T = K Q^T per 16-key block: lane (g, n) ends with keys 16 kb + 4 g + i of query n
        f32x4 s[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
            const int kr = kb * 16 + n;
            const float* krow = tile.k + kr * KS;
#pragma unroll
            for (int s4 = 0; s4 < RS; s4 += 4) {
                const float4 a = *(const float4*)(krow + kpos<R>(kr, (grp * RS + s4) / 4) * 4);
                s[kb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, qreg[s4 + 0], s[kb], 0, 0, 0);
                s[kb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, qreg[s4 + 1], s[kb], 0, 0, 0);
                s[kb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, qreg[s4 + 2], s[kb], 0, 0, 0);
                s[kb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, qreg[s4 + 3], s[kb], 0, 0, 0);
            }
        }
        // causal / ragged-tail mask, only where the tile crosses it
        const bool needs_mask = (p.causal && base + BN - 1 > q0 + off) || base + BN > p.Sk;
        if (needs_mask) {
            const int limit = p.causal ? qrow + off : p.Sk - 1;
            const int lim = limit < p.Sk - 1 ? limit : p.Sk - 1;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int key = base + kb * 16 + 4 * grp + i;
                    if (key > lim) s[kb][i] = -INFINITY;
                }
        }
        float mx = max_f(max_f(max_f(s[0][0], s[0][1]), max_f(s[0][2], s[0][3])),
                         max_f(max_f(s[1][0], s[1][1]), max_f(s[1][2], s[1][3])));
        mx = strided_max<16>(mx);  // over the query's 4 lane groups
        const float mx2 = mx * c;
        // each query moves its own reference only, when its maximum exceeds it by
        // more than 8 (a factor of 256); the branch is taken by the whole wave
        // when any query needs it
        const bool need = mx2 > m_ref + 8.f;
        if (__any(need)) {
            const float alpha = need ? exp2_fast(m_ref - mx2) : 1.f;
            m_ref = need ? mx2 : m_ref;
            lsum *= alpha;
#pragma unroll
            for (int d = 0; d < DBLK; ++d) o[d] *= alpha;
        }
        // a query with no reference yet has seen no visible key: its scores are all
        // -inf here (a wave's first tile can lie past a row's causal limit), and
        // exponentiating against 0 gives them weight 0 instead of NaN
        const float m_use = m_ref == -INFINITY ? 0.f : m_ref;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                s[kb][i] = exp2_fast(fmaf(s[kb][i], c, -m_use));
                lsum += s[kb][i];
            }
        // O^T += V^T P^T: contraction step i of block kb takes keys 16 kb + 4 g + i,
        // which lane group g already holds in register i of its score block
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int d = 0; d < DBLK; ++d) {
                const float* vp = tile.v + (kb * 16 + 4 * grp) * VS + d * 16 + n;
                o[d] = __builtin_amdgcn_mfma_f32_16x16x4f32(vp[0], s[kb][0], o[d], 0, 0, 0);
                o[d] = __builtin_amdgcn_mfma_f32_16x16x4f32(vp[VS], s[kb][1], o[d], 0, 0, 0);
                o[d] = __builtin_amdgcn_mfma_f32_16x16x4f32(vp[2 * VS], s[kb][2], o[d], 0, 0, 0);
                o[d] = __builtin_amdgcn_mfma_f32_16x16x4f32(vp[3 * VS], s[kb][3], o[d], 0, 0, 0);
            }
        wave_lds_sync();  // the tile's operand reads are done before the next store
    }

    // ---- merge the 4 waves' partial results (log-sum-exp rule) and write the rows
    const float ltot = strided_sum<16>(lsum);
    __syncthreads();  // every wave is done with its tile: the LDS becomes the merge area
#pragma unroll
    for (int d = 0; d < DBLK; ++d)
#pragma unroll
        for (int i = 0; i < 4; ++i) sm.merge.o[wave][d * 16 + 4 * grp + i][n] = o[d][i];
    if (grp == 0) {
        sm.merge.m[wave][n] = m_ref;
        sm.merge.l[wave][n] = ltot;
    }
    __syncthreads();
    for (int e = tid; e < kRows * DV; e += kThreads) {
        const int q = e / DV, dd = e % DV;
        if (q0 + q >= p.Sq) break;  // rows only grow with e
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) M = fmaxf(M, sm.merge.m[w][q]);
        float O = 0.f, L = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const float mw = sm.merge.m[w][q];
            if (mw == -INFINITY) continue;  // this wave saw no visible key of the row
            const float ew = exp2_fast(mw - M);
            O = fmaf(ew, sm.merge.o[w][dd][q], O);
            L = fmaf(ew, sm.merge.l[w][q], L);
        }
        og[(size_t)(q0 + q) * DV + dd] = O / L;
    }
}

template <int R, int DV>
static hipError_t run(const PrefillParams& p, hipStream_t st) {
    const long n = (long)((p.Sq + kRows - 1) / kRows) * p.Hq * p.B;
    if (n > 0x7fffffffL) return hipErrorInvalidValue;
    dim3 grid((unsigned)n);
    hipLaunchKernelGGL((prefill_f32_kernel<R, DV>), grid, dim3(kThreads), 0, st, p);
    return hipGetLastError();
}

template <int R>
static hipError_t by_dv(const PrefillParams& p, int DV, hipStream_t st) {
    if (DV == 64) return run<R, 64>(p, st);
    if (DV == 128) return run<R, 128>(p, st);
    return hipErrorInvalidValue;
}

tk_status launch_prefill_f32(const PrefillParams& p, int R, int DV, hipStream_t st) {
    hipError_t e;
    switch (R) {
        case 16: e = by_dv<16>(p, DV, st); break;
        case 32: e = by_dv<32>(p, DV, st); break;
        case 64: e = by_dv<64>(p, DV, st); break;
        case 128: e = by_dv<128>(p, DV, st); break;
        default: return TK_ERR_UNSUPPORTED;
    }
    if (e == hipErrorInvalidValue) return TK_ERR_UNSUPPORTED;
    return e == hipSuccess ? TK_OK : TK_ERR_HIP;
}

}  // namespace tk
