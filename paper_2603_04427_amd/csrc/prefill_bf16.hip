// Thin-key causal prefill attention for gfx950, bf16 inputs, fp32 accumulation.
//
// Prefill is compute-bound (the paper's prefill-roofline appendix): per visible
// (query, key) pair it does 2r FLOPs of selection and 2 d_v FLOPs of value
// transfer, with r < d_v for thin keys. Both products run on the bf16 matrix
// cores (v_mfma_f32_32x32x16_bf16); the softmax runs on the vector ALUs.
//
// Work decomposition
//  * A workgroup is 4 waves. Each wave owns 32 query rows (one 32-column MFMA
//    block; QC = 2 gives it 64 rows, each LDS operand read then feeding two
//    MFMAs) of one query head; the workgroup covers HPW = gcd(G, 4) heads of one
//    KV group and 4 / HPW row blocks, so each K/V tile in LDS serves every wave.
//  * 64-key tiles are double-buffered in LDS and filled straight from global
//    memory (global_load_lds, 16 bytes per lane, issued a whole tile ahead and
//    awaited only before the barrier that publishes the tile), K and V both in their memory
//    layout with the 16-byte chunks of each row XOR-swizzled so that the
//    operand reads below are free of bank conflicts.
//  * Scores are computed transposed, S^T = K Q^T: each lane holds 16 keys of one
//    query per 32-key block, so the row maximum and row sum stay in-lane except
//    for one exchange between the two 32-lane halves (v_permlane32_swap), and
//    P^T leaves the accumulators in the B-operand layout of O^T = V^T P^T. The
//    V^T operand (8 keys of one column per lane) comes from the untransposed V
//    tile through the transposing LDS read ds_read_b64_tr_b16.
//  * Online softmax in the log2 domain (scale * log2(e) applied by one FMA),
//    with a lazy per-row rescale: a row's reference maximum moves only when its
//    maximum exceeds it by more than 8 (a factor of 256). With one query block
//    per wave the row sums run on the matrix core, which the vector softmax
//    leaves idle about half the time: a 16x16x32 product of a 0/1 selector with
//    each bf16 P^T operand adds up exactly the rounded probabilities that feed
//    the value product, in place of 16 vector dot products per tile.
//  * Causal masking only on tiles that cross a wave's diagonal; tiles above it
//    are skipped. Workgroups are ordered so that the query blocks of one KV
//    sequence run together on one XCD (its K/V stays in that XCD's L2),
//    heaviest (longest causal prefix) first.
#include "tk_device.hpp"
#include "tk_internal.hpp"

#include <type_traits>

#include <math.h>

namespace tk {

namespace {

constexpr int kBN = 64;  // keys per tile
constexpr int kXcds = 8;

__host__ __device__ constexpr int gcd4(int g) { return (g % 4 == 0) ? 4 : (g % 2 == 0 ? 2 : 1); }

typedef short v4s __attribute__((ext_vector_type(4)));

// Row swizzle of a tile with W bf16 per row: the 16-byte chunk c of row r is
// stored at chunk position c ^ swz(r).
template <int W, bool IS_V>
__device__ __forceinline__ int swz(int r) {
    constexpr int CPR = W / 8;                                // 16-byte chunks per row
    constexpr int RPL = (256 / (2 * W)) > 0 ? 256 / (2 * W) : 1;  // rows per 256-byte bank line
    if constexpr (IS_V) {
        return (4 * (r / RPL)) & (CPR - 1);
    } else {
        return (r / RPL) & (CPR - 1);
    }
}

template <int R, int DV>
struct Smem {
    uint16_t k[2][kBN * R];
    uint16_t v[2][kBN * DV];
};

// Global->LDS copies of one 64-key K and V tile (global_load_lds, 16 bytes per
// lane, each wave filling 1 KB of consecutive LDS). Which 16-byte chunk of which
// row a lane copies does not depend on the tile, so its byte offset inside a
// tile is computed once (TileLanes); a tile then only adds its first row. Copy
// i of a lane takes the chunk NT i further, i.e. NT / (W / 8) rows further down
// at the same chunk position: the row swizzles repeat with a period that
// divides that step, so copy i's offset is copy 0's plus a constant, which the
// wave-uniform global base absorbs. One offset register per tile is kept.
template <int R, int DV, int NT>
struct TileLanes {
    static constexpr int KC = kBN * R / 8;   // 16-byte chunks in the K tile
    static constexpr int VC = kBN * DV / 8;  // ... and in the V tile
    static constexpr int KL = (KC + NT - 1) / NT;
    static constexpr int VL = (VC + NT - 1) / NT;
    static constexpr int KSTEP = NT / (R / 8);   // rows between a lane's copies i and i + 1
    static constexpr int VSTEP = NT / (DV / 8);
    // swizzle periods in rows: swz<W, false> repeats every RPL * CPR rows,
    // swz<W, true> every RPL * CPR / 4
    static constexpr int KPER = ((256 / (2 * R)) > 0 ? 256 / (2 * R) : 1) * (R / 8);
    static constexpr int VPER = ((256 / (2 * DV)) > 0 ? 256 / (2 * DV) : 1) * (DV / 8) / 4;
    static_assert(KL == 1 || KSTEP % KPER == 0, "K copy offsets are not a constant stride apart");
    static_assert(VL == 1 || VSTEP % VPER == 0, "V copy offsets are not a constant stride apart");
    uint32_t k_off;  // byte offset (in the tile) of this lane's first K chunk
    uint32_t v_off;
    int tid_;

    __device__ __forceinline__ explicit TileLanes(int tid) : tid_(tid) {
        const int kr = tid / (R / 8), kp = tid % (R / 8);
        k_off = (uint32_t)((kr * R + (kp ^ swz<R, false>(kr)) * 8) * 2);
        const int vr = tid / (DV / 8), vp = tid % (DV / 8);
        v_off = (uint32_t)((vr * DV + (vp ^ swz<DV, true>(vr)) * 8) * 2);
    }
    // tile rows of the chunks, recomputed (needed only for a ragged last tile)
    __device__ __forceinline__ int k_row(int i) const { return (tid_ + i * NT) / (R / 8); }
    __device__ __forceinline__ int v_row(int i) const { return (tid_ + i * NT) / (DV / 8); }
};

// Issue the copies of the tile starting at key `base` (wave `wave` copies its
// 1 KB slices). A full tile needs no vector arithmetic: the global base and the
// LDS destination are wave-uniform and the lane offset is precomputed. Rows
// at or past Sk (only in a ragged last tile) re-read row Sk - 1: finite values,
// masked later.
template <int R, int DV, int NT>
__device__ __forceinline__ void load_tile(const TileLanes<R, DV, NT>& tl, uint16_t* ks, uint16_t* vs,
                                          const uint16_t* kg, const uint16_t* vg, int base, int Sk, int wave) {
    using T = TileLanes<R, DV, NT>;
    const int wave_base = wave * 64;
    const char* kt = (const char*)(kg + (size_t)base * R);
    const char* vt = (const char*)(vg + (size_t)base * DV);
    if (base + kBN <= Sk) {  // workgroup-uniform
#pragma unroll
        for (int i = 0; i < T::KL; ++i) {
            if (T::KC % NT != 0 && wave_base + i * NT >= T::KC) break;
            copy16_to_lds(kt + i * T::KSTEP * R * 2, tl.k_off, ks + (wave_base + i * NT) * 8);
        }
#pragma unroll
        for (int i = 0; i < T::VL; ++i) {
            if (T::VC % NT != 0 && wave_base + i * NT >= T::VC) break;
            copy16_to_lds(vt + i * T::VSTEP * DV * 2, tl.v_off, vs + (wave_base + i * NT) * 8);
        }
        return;
    }
    // A ragged tile clamps rows past the end to row `last` by lowering the
    // offset. The copy's vector offset is unsigned, so here every copy keeps the
    // tile's own base and adds its stride to the offset: the clamped offset then
    // stays non-negative even where `last` lies above copy i's first row.
    int last = Sk - base - 1;
    // opaque to the loop's induction analysis: otherwise the compiler keeps the
    // clamped offsets as induction variables updated on every tile, though
    // only a ragged last tile uses them
    asm volatile("" : "+s"(last));
#pragma unroll
    for (int i = 0; i < T::KL; ++i) {
        if (T::KC % NT != 0 && wave_base + i * NT >= T::KC) break;
        const int kr = tl.k_row(i);
        const uint32_t oi = tl.k_off + (uint32_t)(i * T::KSTEP * R * 2);
        const uint32_t off = kr > last ? oi - (uint32_t)((kr - last) * R * 2) : oi;
        copy16_to_lds(kt, off, ks + (wave_base + i * NT) * 8);
    }
#pragma unroll
    for (int i = 0; i < T::VL; ++i) {
        if (T::VC % NT != 0 && wave_base + i * NT >= T::VC) break;
        const int vr = tl.v_row(i);
        const uint32_t oi = tl.v_off + (uint32_t)(i * T::VSTEP * DV * 2);
        const uint32_t off = vr > last ? oi - (uint32_t)((vr - last) * DV * 2) : oi;
        copy16_to_lds(vt, off, vs + (wave_base + i * NT) * 8);
    }
}

// exp2(s * c - m) for the 16 keys of k-step q of one 32-query block (accumulator
// registers 8 (q % 2) .. + 7 of key block q / 2), rounded to a bf16 B operand of
// O^T = V^T P^T; the row-sum share accumulates the same rounded values.
template <bool SUM = true>
__device__ __forceinline__ bf16x8 prob_step(const f32x16 (&s)[2], int q, float m, float c, float& lsum) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float p0 = exp2_fast(fmaf(s[q >> 1][8 * (q & 1) + 2 * i], c, -m));
        const float p1 = exp2_fast(fmaf(s[q >> 1][8 * (q & 1) + 2 * i + 1], c, -m));
        w[i] = pack_bf16(p0, p1);
        if constexpr (SUM) lsum = add_bf16_pair(w[i], lsum);
    }
    return __builtin_bit_cast(bf16x8, make_uint4(w[0], w[1], w[2], w[3]));
}

// Transposing LDS read of 4 bf16 (ds_read_b64_tr_b16) at byte offset `off`.
__device__ __forceinline__ v4s tr_read(const uint16_t* tile, uint32_t off) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) v4s*)((const char*)tile + off));
}

// The V^T operand of k-step q, column block d: lane (half h, column i) needs
// V[16q + 4h + j][32d + i] (slots 0-3) and V[16q + 8 + 4h + j][32d + i] (slots
// 4-7), j = 0..3, gathered by two transposing reads in which source lane L of
// each 16-lane group points at row k0 + L/4, columns d0 + 4 (L % 4) .. + 3.
// `vbase` is the lane's byte offset for q = 0 (the swizzle term does not depend
// on q), so k-step q adds 16 q rows.
template <int DV>
__device__ __forceinline__ bf16x8 vt_operand(const uint16_t* vs, uint32_t vbase, int q) {
    const v4s lo = tr_read(vs, vbase + 16 * q * DV * 2);
    const v4s hi = tr_read(vs, vbase + (16 * q + 8) * DV * 2);
    bf16x8 a;
    a[0] = lo[0];
    a[1] = lo[1];
    a[2] = lo[2];
    a[3] = lo[3];
    a[4] = hi[0];
    a[5] = hi[1];
    a[6] = hi[2];
    a[7] = hi[3];
    return a;
}

}  // namespace

// QC: 32-query column blocks per wave (1 or 2); NW: waves per workgroup.
template <int R, int DV, int QC, int NW>
__global__ __launch_bounds__(64 * NW, QC == 1 ? (R <= 32 ? 3 : 2) : 1) void prefill_bf16_kernel(const PrefillParams p,
                                                                                     int n_groups) {
    constexpr int KSTEPS = R / 16;  // MFMA K-steps of the score product
    constexpr int DBLK = DV / 32;   // 32-row blocks of O^T
    constexpr int NT = 64 * NW;
    __shared__ Smem<R, DV> sm;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = lane >> 5, col = lane & 31;

    // ---- workgroup -> (KV sequence, query block), XCD-aware and heaviest first
    const int HPW = gcd4(p.G);
    const int RB = NW / HPW;
    const int BM = 32 * QC * RB;
    const int nqb = (p.Sq + BM - 1) / BM;
    const int per_xcd = (n_groups + kXcds - 1) / kXcds;
    const int logical = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    if (logical >= n_groups) return;
    const int pair = logical / nqb, rank = logical % nqb;
    const int qb = p.causal ? nqb - 1 - rank : rank;
    const int groups_per_kv = p.G / HPW;
    const int b = pair / (p.Hkv * groups_per_kv);
    const int gy = pair % (p.Hkv * groups_per_kv);
    const int g = gy / groups_per_kv;
    const int h = g * p.G + (gy % groups_per_kv) * HPW + wave % HPW;
    const int q0 = qb * BM;
    const int qw0 = q0 + (wave / HPW) * 32 * QC;  // first row of this wave
    const int off = p.Sk - p.Sq;             // bottom-right causal alignment

    const uint16_t* qg = (const uint16_t*)p.q + ((size_t)b * p.Hq + h) * p.Sq * R;
    const uint16_t* kg = (const uint16_t*)p.k + ((size_t)b * p.Hkv + g) * p.Sk * R;
    const uint16_t* vg = (const uint16_t*)p.v + ((size_t)b * p.Hkv + g) * p.Sk * DV;
    uint16_t* og = (uint16_t*)p.o + ((size_t)b * p.Hq + h) * p.Sq * DV;

    int key_end = p.Sk;
    if (p.causal) {
        const int last = q0 + BM - 1 + off + 1;
        key_end = last < key_end ? last : key_end;
    }
    const int ntiles = (key_end + kBN - 1) / kBN;
    const TileLanes<R, DV, NT> tl(tid);
    load_tile<R, DV, NT>(tl, sm.k[0], sm.v[0], kg, vg, 0, p.Sk, wave);

    // Q^T operands: column block qc holds query rows qw0 + 32 qc + col, dims 16m + 8 half .. +7
    bf16x8 qreg[QC][KSTEPS];
#pragma unroll
    for (int qc = 0; qc < QC; ++qc) {
        const int qrow = qw0 + 32 * qc + col;
#pragma unroll
        for (int m = 0; m < KSTEPS; ++m) {
            const uint4 w =
                qrow < p.Sq ? *(const uint4*)(qg + (size_t)qrow * R + 16 * m + 8 * half) : make_uint4(0, 0, 0, 0);
            qreg[qc][m] = __builtin_bit_cast(bf16x8, w);
        }
    }
    const int wave_last_key = p.causal ? qw0 + 32 * QC - 1 + off : p.Sk - 1;  // last key any row of the wave sees

    f32x16 o[QC][DBLK];
#pragma unroll
    for (int qc = 0; qc < QC; ++qc)
#pragma unroll
        for (int d = 0; d < DBLK; ++d)
#pragma unroll
            for (int v = 0; v < 16; ++v) o[qc][d][v] = 0.f;
    float m_ref[QC], lsum[QC];  // running reference maxima (log2 domain); this lane's half of each row sum
#pragma unroll
    for (int qc = 0; qc < QC; ++qc) {
        m_ref[qc] = -INFINITY;
        lsum[qc] = 0.f;
    }
    const float c = p.qscale;
    // Row sums on the matrix core (one query block per wave): a 16x16x32 product
    // of a 0/1 selector with each P^T operand. Lanes 0 and 32 of the selector
    // pick the keys a query's two lane halves hold into row 0 (query n), lanes 17
    // and 49 into row 1 (query n + 16); lanes 0..15 of the accumulator then hold
    // the sums of queries n (register 0) and n + 16 (register 1).
    constexpr bool MSUM = QC == 1;
    f32x4 lacc = {0.f, 0.f, 0.f, 0.f};
    bf16x8 sel;
    {
        const uint32_t one = (lane == 0 || lane == 32 || lane == 17 || lane == 49) ? 0x3F803F80u : 0u;
        sel = __builtin_bit_cast(bf16x8, make_uint4(one, one, one, one));
    }

    // Lane byte offsets of the LDS operands. The row swizzles reduce to lane
    // constants here: for K rows kb*32 + col the swizzle term depends on col
    // only, for the V rows read below on lane % 16 only.
    uint32_t kaddr[KSTEPS];
#pragma unroll
    for (int m = 0; m < KSTEPS; ++m) kaddr[m] = (uint32_t)((col * R + (((2 * m + half) ^ swz<R, false>(col)) * 8)) * 2);
    uint32_t vaddr[DBLK];
    {
        const int li = lane & 15, grp = lane >> 4;
        const int sv = swz<DV, true>(li >> 2);
#pragma unroll
        for (int d = 0; d < DBLK; ++d) {
            const int col0 = 32 * d + 16 * (grp & 1) + 4 * (li & 3);
            const int r1 = 4 * half + (li >> 2);
            vaddr[d] = (uint32_t)((r1 * DV + (((col0 >> 3) ^ sv) * 8) + (col0 & 7)) * 2);
        }
    }
    wait_loads();
    // the same wait as a builtin, so that the compiler knows the query loads
    // have landed and adds no wait of its own inside the tile loop (vmcnt 0;
    // expcnt and lgkmcnt at their maxima)
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();

    // the loop over key tiles, two tiles per iteration, so that the double buffer
    // each tile uses is a compile-time constant and its LDS addresses take
    // immediate offsets
    auto tile_step = [&](auto cur_c, int t) {
        constexpr int cur = decltype(cur_c)::value;
        const int base = t * kBN;
        if (t + 1 < ntiles) load_tile<R, DV, NT>(tl, sm.k[cur ^ 1], sm.v[cur ^ 1], kg, vg, base + kBN, p.Sk, wave);

        if (base <= wave_last_key) {
            const uint16_t* ks = sm.k[cur];
            const uint16_t* vs = sm.v[cur];
            // ---- S^T = K Q^T: two 32-key blocks x two query blocks
            f32x16 s[QC][2];
#pragma unroll
            for (int qc = 0; qc < QC; ++qc)
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int v = 0; v < 16; ++v) s[qc][kb][v] = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
                for (int m = 0; m < KSTEPS; ++m) {
                    const bf16x8 a = *(const bf16x8*)((const char*)ks + kaddr[m] + kb * 32 * R * 2);
#pragma unroll
                    for (int qc = 0; qc < QC; ++qc)
                        s[qc][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[qc][m], s[qc][kb], 0, 0, 0);
                }
            }
            // ---- causal / ragged-tail mask, only where the tile crosses it
            const bool needs_mask = (p.causal && base + kBN - 1 > qw0 + off) || base + kBN > p.Sk;
            if (needs_mask) {
#pragma unroll
                for (int qc = 0; qc < QC; ++qc) {
                    const int qrow = qw0 + 32 * qc + col;
                    int lim = p.causal ? qrow + off : p.Sk - 1;
                    lim = lim < p.Sk - 1 ? lim : p.Sk - 1;
#pragma unroll
                    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                        for (int v = 0; v < 16; ++v) {
                            const int key = base + kb * 32 + 8 * (v >> 2) + 4 * half + (v & 3);
                            if (key > lim) s[qc][kb][v] = -INFINITY;
                        }
                }
            }
            // ---- row maxima (v_maximum3_f32) and lazy rescale for each query block
            // (the only branches)
#pragma unroll
            for (int qc = 0; qc < QC; ++qc) {
                float mx = s[qc][0][0];
#pragma unroll
                for (int v = 1; v < 16; ++v) mx = max_f(mx, s[qc][0][v]);
#pragma unroll
                for (int v = 0; v < 16; ++v) mx = max_f(mx, s[qc][1][v]);
                mx = xor32_max(mx);
                const float mx2 = mx * c;
                // each row moves its own reference; the branch is taken by the whole
                // wave when any row needs it
                const bool need = mx2 > m_ref[qc] + 8.f;
                if (__any(need)) {
                    const float alpha = need ? exp2_fast(m_ref[qc] - mx2) : 1.f;
                    m_ref[qc] = need ? mx2 : m_ref[qc];
                    lsum[qc] *= alpha;
                    if constexpr (MSUM) {
                        const float alpha_hi = __shfl_xor(alpha, 16);  // query n + 16's factor
                        lacc[0] *= alpha;
                        lacc[1] *= alpha_hi;
                    }
#pragma unroll
                    for (int d = 0; d < DBLK; ++d)
#pragma unroll
                        for (int v = 0; v < 16; ++v) o[qc][d][v] *= alpha;
                }
            }
            // ---- probabilities and O^T += V^T P^T, k-step by k-step. Each V^T operand
            // is read once for both query blocks, one k-step ahead; within a k-step
            // the matrix operations of query block 0 are interleaved with the
            // vector work producing block 1's probabilities, and those of block 1
            // with block 0's next probabilities, so one wave keeps both pipes busy
            bf16x8 va[DBLK];
#pragma unroll
            for (int d = 0; d < DBLK; ++d) va[d] = vt_operand<DV>(vs, vaddr[d], 0);
            bf16x8 p0 = prob_step<!MSUM>(s[0], 0, m_ref[0], c, lsum[0]);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                __builtin_amdgcn_sched_barrier(0);
                bf16x8 vb[DBLK];
                if (q < 3) {
#pragma unroll
                    for (int d = 0; d < DBLK; ++d) vb[d] = vt_operand<DV>(vs, vaddr[d], q + 1);
                }
                bf16x8 p1 = p0;
                if constexpr (QC == 2) p1 = prob_step(s[QC - 1], q, m_ref[QC - 1], c, lsum[QC - 1]);
                bf16x8 p0n = p0;
                if (q < 3) p0n = prob_step<!MSUM>(s[0], q + 1, m_ref[0], c, lsum[0]);
#pragma unroll
                for (int d = 0; d < DBLK; ++d)
                    o[0][d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[d], p0, o[0][d], 0, 0, 0);
                if constexpr (MSUM) lacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel, p0, lacc, 0, 0, 0);
                if constexpr (QC == 2) {
#pragma unroll
                    for (int d = 0; d < DBLK; ++d)
                        o[QC - 1][d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[d], p1, o[QC - 1][d], 0, 0, 0);
                }
                // schedule: operand reads first, then one MFMA per few vector ops
                __builtin_amdgcn_sched_group_barrier(0x100, 4 * DBLK, 0);
#pragma unroll
                for (int i = 0; i < QC * DBLK + (MSUM ? 1 : 0); ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x402, MSUM ? 4 : 6, 0);
                }
                if (q < 3) {
                    p0 = p0n;
#pragma unroll
                    for (int d = 0; d < DBLK; ++d) va[d] = vb[d];
                }
            }
        }

        if (t + 1 < ntiles) wait_loads();  // this wave's part of the next tile has landed
        __syncthreads();
    };
    int t = 0;
    for (; t + 1 < ntiles; t += 2) {
        tile_step(std::integral_constant<int, 0>{}, t);
        tile_step(std::integral_constant<int, 1>{}, t + 1);
    }
    if (t < ntiles) tile_step(std::integral_constant<int, 0>{}, t);

    // ---- epilogue: normalise and store bf16 rows (and, when asked, the row's
    // log-sum-exp: the reference maximum plus log2 of the sum, in natural log)
#pragma unroll
    for (int qc = 0; qc < QC; ++qc) {
        float ltot;
        if constexpr (MSUM) {
            const float a0 = __shfl(lacc[0], col & 15);
            const float a1 = __shfl(lacc[1], col & 15);
            ltot = col < 16 ? a0 : a1;
        } else {
            ltot = xor32_sum(lsum[qc]);
        }
        const float inv = 1.f / ltot;
        const int qrow = qw0 + 32 * qc + col;
        if (p.lse != nullptr && half == 0 && qrow < p.Sq)
            p.lse[((size_t)b * p.Hq + h) * p.Sq + qrow] = (m_ref[qc] + __builtin_amdgcn_logf(ltot)) * kLn2;
        if (qrow < p.Sq) {
            uint16_t* orow = og + (size_t)qrow * DV;
#pragma unroll
            for (int d = 0; d < DBLK; ++d)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    uint2 w;
                    w.x = pack_bf16(o[qc][d][4 * j] * inv, o[qc][d][4 * j + 1] * inv);
                    w.y = pack_bf16(o[qc][d][4 * j + 2] * inv, o[qc][d][4 * j + 3] * inv);
                    *(uint2*)(orow + d * 32 + 8 * j + 4 * half) = w;
                }
        }
    }
}

template <int R, int DV, int QC, int NW>
static hipError_t run(const PrefillParams& p, hipStream_t st) {
    const int HPW = gcd4(p.G);
    const int BM = 32 * QC * (NW / HPW);
    const long nqb = (p.Sq + BM - 1) / BM;
    const long groups = nqb * p.Hkv * (p.G / HPW) * p.B;
    const long launched = (groups + kXcds - 1) / kXcds * kXcds;
    if (launched > 0x7fffffffL) return hipErrorInvalidValue;
    hipLaunchKernelGGL((prefill_bf16_kernel<R, DV, QC, NW>), dim3((unsigned)launched), dim3(64 * NW), 0, st, p,
                       (int)groups);
    return hipGetLastError();
}

#ifndef TK_PREFILL_QC
#define TK_PREFILL_QC 1
#endif
#ifndef TK_PREFILL_WAVES
#define TK_PREFILL_WAVES 4
#endif

template <int R, int DV>
static hipError_t run(const PrefillParams& p, hipStream_t st) {
    return run<R, DV, TK_PREFILL_QC, TK_PREFILL_WAVES>(p, st);
}

template <int R>
static hipError_t by_dv(const PrefillParams& p, int DV, hipStream_t st) {
    if (DV == 64) return run<R, 64>(p, st);
    if (DV == 128) return run<R, 128>(p, st);
    return hipErrorInvalidValue;
}

tk_status launch_prefill_bf16(const PrefillParams& p, int R, int DV, hipStream_t st) {
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
