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
// longest first, so the round-robin dispatch deals every XCD the same mix.
//
// Inside a wave: transposed scores S^T = K Q^T per 16-key block, so lane (g, n)
// of lane group g = lane / 16 serves query n = lane % 16, and O^T = V^T P^T.
// Each instruction contracts 4 indices, one per lane group, so:
//  * the score product walks r in R/4 steps, lane group g covering dims
//    [g R/4, (g+1) R/4) (contiguous in the K row, read 16 bytes at a time);
//  * the value product takes, in step i of a key block, keys 4 g + i: the keys
//    whose scores lane group g already holds in accumulator register i, so P^T
//    is used in place with no repacking. V is stored transposed ([d_v][keys]
//    fp32, natural key order) so one 16-byte read gives a lane the operands of
//    four steps.
// Row maxima and sums reduce over the four lane groups of a query (lane
// n, n + 16, n + 32, n + 48). A wave loads its next tile into registers while
// it computes the current one.
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
// the workgroup's four tiles take 45 KB of LDS, so three workgroups share a CU
// and one wave's softmax overlaps another's matrix products (with 64-key tiles
// only one workgroup fits and a wave's dependent score -> softmax -> value
// chain leaves its matrix core idle for about 40 % of a tile).
template <int R, int DV>
struct alignas(16) WaveTile {
    static constexpr int BN = 32;
    static constexpr int KB = BN / 32;  // 32-key blocks per tile
    static constexpr int KS = R + 4;    // floats per K row in LDS (16-byte pad)
    static constexpr int VS = BN + 4;   // floats per transposed V row
    float k[BN * KS];
    float vt[DV * VS];
};

// One tile of one wave in registers: 16-byte K chunks and 4-key x 4-column V quads.
template <int R, int DV>
struct WaveRegs {
    static constexpr int BN = WaveTile<R, DV>::BN;
    static constexpr int KCH = BN * R / 4;
    static constexpr int VQ = (BN / 4) * (DV / 4);
    static_assert(KCH % 64 == 0 && VQ % 64 == 0, "tile does not divide over the lanes");
    static constexpr int KL = KCH / 64;
    static constexpr int VL = VQ / 64;
    float4 k[KL];
    float4 v[VL][4];
};

// Keys at or past Sk (only in a ragged last tile) load as zeros; they are masked.
// A full tile (the wave-uniform common case) loads without per-lane tests.
template <int R, int DV>
__device__ __forceinline__ void load_tile(WaveRegs<R, DV>& t, const float* kg, const float* vg, int base, int Sk,
                                          int lane) {
    using W = WaveRegs<R, DV>;
    constexpr int CPR = R / 4;
    if (base + W::BN <= Sk) {
#pragma unroll
        for (int i = 0; i < W::KL; ++i) {
            const int c = lane + 64 * i;
            t.k[i] = *(const float4*)(kg + (size_t)(base + c / CPR) * R + (c % CPR) * 4);
        }
#pragma unroll
        for (int i = 0; i < W::VL; ++i) {
            const int qd = lane + 64 * i;
            const int kq = qd % (W::BN / 4), dc = qd / (W::BN / 4);
#pragma unroll
            for (int j = 0; j < 4; ++j) t.v[i][j] = *(const float4*)(vg + (size_t)(base + 4 * kq + j) * DV + dc * 4);
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < W::KL; ++i) {
        const int c = lane + 64 * i;
        const int row = c / CPR, part = c % CPR;
        t.k[i] = base + row < Sk ? *(const float4*)(kg + (size_t)(base + row) * R + part * 4)
                                 : make_float4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < W::VL; ++i) {
        const int qd = lane + 64 * i;
        const int kq = qd % (W::BN / 4), dc = qd / (W::BN / 4);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int key = base + 4 * kq + j;
            t.v[i][j] = key < Sk ? *(const float4*)(vg + (size_t)key * DV + dc * 4) : make_float4(0, 0, 0, 0);
        }
    }
}

template <int R, int DV>
__device__ __forceinline__ void store_tile(const WaveRegs<R, DV>& t, WaveTile<R, DV>& tile, int lane) {
    using W = WaveRegs<R, DV>;
    using T = WaveTile<R, DV>;
    constexpr int CPR = R / 4;
#pragma unroll
    for (int i = 0; i < W::KL; ++i) {
        const int c = lane + 64 * i;
        const int row = c / CPR, part = c % CPR;
        *(float4*)(tile.k + row * T::KS + part * 4) = t.k[i];
    }
#pragma unroll
    for (int i = 0; i < W::VL; ++i) {
        const int qd = lane + 64 * i;
        const int kq = qd % (W::BN / 4), dc = qd / (W::BN / 4);
        const float4* x = t.v[i];
        // 4 keys x 4 columns -> 4 rows of V^T, 4 consecutive keys each
        *(float4*)(tile.vt + (dc * 4 + 0) * T::VS + 4 * kq) = make_float4(x[0].x, x[1].x, x[2].x, x[3].x);
        *(float4*)(tile.vt + (dc * 4 + 1) * T::VS + 4 * kq) = make_float4(x[0].y, x[1].y, x[2].y, x[3].y);
        *(float4*)(tile.vt + (dc * 4 + 2) * T::VS + 4 * kq) = make_float4(x[0].z, x[1].z, x[2].z, x[3].z);
        *(float4*)(tile.vt + (dc * 4 + 3) * T::VS + 4 * kq) = make_float4(x[0].w, x[1].w, x[2].w, x[3].w);
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
    const int lane = tid & 63, wave = tid >> 6;
    const int grp = lane >> 4, n = lane & 15;  // lane group, and the query (B column) the lane serves

    // workgroup -> (query block, head, sequence): ranked by causal prefix length,
    // longest first, with the heads and sequences of one rank adjacent, so that the
    // round-robin dispatch over the XCDs deals every XCD the same mix of long and
    // short blocks
    const int nqb = (p.Sq + kRows - 1) / kRows;
    const int rank = (int)(blockIdx.x / ((unsigned)p.Hq * p.B));
    const int hb = (int)(blockIdx.x % ((unsigned)p.Hq * p.B));
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
            const float* krow = tile.k + (kb * 16 + n) * KS + grp * RS;
#pragma unroll
            for (int s4 = 0; s4 < RS; s4 += 4) {
                const float4 a = *(const float4*)(krow + s4);
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
        float mx = fmaxf(fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3])),
                         fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
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
                const float4 a = *(const float4*)(tile.vt + (d * 16 + n) * VS + kb * 16 + 4 * grp);
                o[d] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, s[kb][0], o[d], 0, 0, 0);
                o[d] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, s[kb][1], o[d], 0, 0, 0);
                o[d] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, s[kb][2], o[d], 0, 0, 0);
                o[d] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, s[kb][3], o[d], 0, 0, 0);
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
