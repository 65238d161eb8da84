// Thin-key prefill attention for gfx950 with fp32 inputs and fp32 matrix cores
// (v_mfma_f32_32x32x2f32), for callers that need fp32 accuracy (bf16 operands
// would not hold a 1e-4 error bound).
//
// Work decomposition. The fp32 matrix instruction does 4096 FLOPs in 64 cycles,
// so a 32-row query block against a long causal prefix is a long serial chain.
// A workgroup therefore holds ONE block of 32 query rows of one head, and its 4
// waves split that block's key tiles among themselves (wave w takes tiles w,
// w + 4, ...), each wave with its own tile in LDS and its own online-softmax
// state; the 4 partial results are merged in LDS with the log-sum-exp rule at
// the end. The longest chain is a quarter of the block's tiles, and a prefill
// has one workgroup per (32 query rows, head).
//
// Inside a wave, as in the bf16 kernel: transposed scores S^T = K Q^T so each
// lane owns one query column, and O^T = V^T P^T. With K = 2 per instruction
// each 32-lane half contributes one contraction index per step, so:
//  * the score product walks r in R/2 steps, lane half h covering dims
//    [h R/2, (h+1) R/2) (contiguous in the K row, read 16 bytes at a time);
//  * the value product walks the 32 keys of a block in 16 steps, lane half h
//    supplying the key that its accumulator register already holds, so P^T is
//    used in place with no repacking. V is stored transposed ([d_v][keys] fp32,
//    natural key order) so four consecutive steps' operands are one 16-byte read.
// A wave loads its next tile into registers while it computes the current one.
#include "tk_device.hpp"
#include "tk_internal.hpp"

#include <math.h>

namespace tk {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kRows = 32;  // query rows per workgroup

// Keys per tile: one 32-key block. A wave's tile then costs 32 (R + DV) / 64
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
    constexpr int HR = R / 2;  // score-product steps (dims per lane half)
    constexpr int DBLK = DV / 32;
    constexpr int BN = T::BN, KB = T::KB, KS = T::KS, VS = T::VS;
    __shared__ Smem<R, DV> sm;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int half = lane >> 5, col = lane & 31;

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

    const int qrow = q0 + col;
    float qreg[HR];
#pragma unroll
    for (int s = 0; s < HR; ++s) qreg[s] = qrow < p.Sq ? qg[(size_t)qrow * R + half * HR + s] : 0.f;

    int key_end = p.Sk;
    if (p.causal) {
        const int last = q0 + kRows + off;  // one past the last key the block's last row sees
        key_end = last < key_end ? last : key_end;
    }
    const int ntiles = (key_end + BN - 1) / BN;

    f32x16 o[DBLK];
#pragma unroll
    for (int d = 0; d < DBLK; ++d)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[d][v] = 0.f;
    float m_ref = -INFINITY;  // this row's reference maximum (log2 domain)
    float lsum = 0.f;         // this lane half's share of the row sum
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

        f32x16 s[KB];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
            for (int v = 0; v < 16; ++v) s[kb][v] = 0.f;
            const float* krow = tile.k + (kb * 32 + col) * KS + half * HR;
#pragma unroll
            for (int s4 = 0; s4 < HR; s4 += 4) {
                const float4 a = *(const float4*)(krow + s4);
                s[kb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.x, qreg[s4 + 0], s[kb], 0, 0, 0);
                s[kb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.y, qreg[s4 + 1], s[kb], 0, 0, 0);
                s[kb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.z, qreg[s4 + 2], s[kb], 0, 0, 0);
                s[kb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.w, qreg[s4 + 3], s[kb], 0, 0, 0);
            }
        }
        // causal / ragged-tail mask, only where the tile crosses it
        const bool needs_mask = (p.causal && base + BN - 1 > q0 + off) || base + BN > p.Sk;
        if (needs_mask) {
            const int limit = p.causal ? qrow + off : p.Sk - 1;
            const int lim = limit < p.Sk - 1 ? limit : p.Sk - 1;
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int key = base + kb * 32 + 8 * (v >> 2) + 4 * half + (v & 3);
                    if (key > lim) s[kb][v] = -INFINITY;
                }
        }
        float mx = s[0][0];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[kb][v]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float mx2 = mx * c;
        // each row moves its own reference only, when its maximum exceeds it by
        // more than 8 (a factor of 256); the branch is taken by the whole wave
        // when any row needs it
        const bool need = mx2 > m_ref + 8.f;
        if (__any(need)) {
            const float alpha = need ? exp2_fast(m_ref - mx2) : 1.f;
            m_ref = need ? mx2 : m_ref;
            lsum *= alpha;
#pragma unroll
            for (int d = 0; d < DBLK; ++d)
#pragma unroll
                for (int v = 0; v < 16; ++v) o[d][v] *= alpha;
        }
        // a row with no reference yet has seen no visible key: its scores are all
        // -inf here (a wave's first tile can lie past a row's causal limit), and
        // exponentiating against 0 gives them weight 0 instead of NaN
        const float m_use = m_ref == -INFINITY ? 0.f : m_ref;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                s[kb][v] = exp2_fast(fmaf(s[kb][v], c, -m_use));
                lsum += s[kb][v];
            }
        // O^T += V^T P^T, one key per lane half per step
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int d = 0; d < DBLK; ++d) {
                const float* vrow = tile.vt + (d * 32 + col) * VS + kb * 32 + 4 * half;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float4 a = *(const float4*)(vrow + 8 * j);
                    o[d] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.x, s[kb][4 * j + 0], o[d], 0, 0, 0);
                    o[d] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.y, s[kb][4 * j + 1], o[d], 0, 0, 0);
                    o[d] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.z, s[kb][4 * j + 2], o[d], 0, 0, 0);
                    o[d] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.w, s[kb][4 * j + 3], o[d], 0, 0, 0);
                }
            }
        wave_lds_sync();  // the tile's operand reads are done before the next store
    }

    // ---- merge the 4 waves' partial results (log-sum-exp rule) and write the rows
    const float ltot = lsum + __shfl_xor(lsum, 32);
    __syncthreads();  // every wave is done with its tile: the LDS becomes the merge area
#pragma unroll
    for (int d = 0; d < DBLK; ++d)
#pragma unroll
        for (int v = 0; v < 16; ++v) sm.merge.o[wave][d * 32 + 8 * (v >> 2) + 4 * half + (v & 3)][col] = o[d][v];
    if (half == 0) {
        sm.merge.m[wave][col] = m_ref;
        sm.merge.l[wave][col] = ltot;
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
