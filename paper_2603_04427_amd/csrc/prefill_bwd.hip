// Backward pass of the thin-key causal prefill for gfx950 (bf16 in and out,
// fp32 accumulation): the gradients that training thin-key models needs.
//
// With the forward's log-sum-exp L of each row and D = rowsum(dO * O):
//     P  = exp(scale S - L),  S = Q K^T      (r-wide contraction)
//     dP = dO V^T                            (d_v-wide contraction)
//     dS = P * (dP - D)
//     dV = P^T dO,  dK = scale dS^T Q,  dQ = scale dS K
// summed over the query heads of each KV group for dK and dV.
//
// Two kernels, no atomics, so results are bitwise reproducible:
//  * bwd_dq_kernel, query-major (the forward's decomposition): a wave owns 32
//    query rows and walks the key tiles. Scores are transposed, S^T = K Q^T and
//    dP^T = V dO^T, so a lane owns one query column and its L and D stay in the
//    lane; dQ^T = K^T dS^T takes K^T from the K tile through the transposing LDS
//    read and dS^T straight from the accumulators. It also writes D, computed
//    from the lane's own dO and O slices.
//  * bwd_dkdv_kernel, key-major: a wave owns 32 keys (K and V rows in
//    registers) and walks the query tiles of every head of the group, from the
//    last tile down to its diagonal with the heads innermost, so that all key
//    blocks of a KV sequence read the same Q and dO tile at about the same
//    time (one fetch into the XCD's L2 serves them all). Scores are
//    S = Q K^T, so a lane owns one key and P and dS leave the accumulators
//    already in the A-operand layout of dV = P^T dO and dK = dS^T Q, whose B
//    operands (dO and Q with 8 query rows per lane) come from the transposing
//    read of the dO and Q tiles.
// Within a 16-wide contraction step the accumulators hold rows 4h + j and
// 8 + 4h + j (lane half h, j = 0..3); the transposing reads gather the other
// operand in that same order, so no repacking is needed.
#include "tk_device.hpp"
#include "tk_internal.hpp"

#include <math.h>

namespace tk {

namespace {

constexpr int kT = 64;  // keys (dq kernel) or query rows (dk/dv kernel) per LDS tile
constexpr int kXcds = 8;
constexpr int kThreads = 256;

__host__ __device__ constexpr int gcd4(int g) { return (g % 4 == 0) ? 4 : (g % 2 == 0 ? 2 : 1); }

typedef short v4s __attribute__((ext_vector_type(4)));

// Row swizzle of an LDS tile with W bf16 per row: 16-byte chunk c of row r is
// stored at chunk position c ^ swz(r). Every tile here is read two ways: by rows
// (16 consecutive rows, one chunk each, per 16 lanes) and through the
// transposing read (4 consecutive rows from a multiple of 4, 4 consecutive
// chunks each, per 32 lanes). With 256-byte bank lines both are conflict-free
// when swz is a bijection over the rows sharing a bank-line position and moves
// the 4-chunk groups of 4 consecutive rows to distinct banks.
template <int W>
__device__ __forceinline__ int swz(int r) {
    if constexpr (W == 32) {
        return (r >> 2) & 3;  // 4 rows per bank line: the transposed read is conflict-free anyway
    } else if constexpr (W == 64) {
        const int x = (r >> 1) & 7;  // 2 rows per bank line
        return ((x & 1) << 2) | (x >> 1);
    } else {
        return ((r & 3) << 2) | ((r >> 2) & 3);  // one row per bank line
    }
}
// Byte offset of element (row, col) in a swizzled tile, col a multiple of 4.
template <int W>
__device__ __forceinline__ uint32_t toff(int row, int col) {
    return (uint32_t)((row * W + (((col >> 3) ^ swz<W>(row)) * 8) + (col & 7)) * 2);
}

// The 8 bf16 of a row-major operand: row `row`, columns col .. col + 7.
template <int W>
__device__ __forceinline__ bf16x8 row_operand(const uint16_t* tile, int row, int col) {
    return *(const bf16x8*)((const char*)tile + toff<W>(row, col));
}

__device__ __forceinline__ v4s tr_read(const uint16_t* tile, uint32_t off) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) v4s*)((const char*)tile + off));
}

// The transposed operand of a 16-row contraction step starting at row r0, for
// the 32 columns c0 .. c0 + 31: lane (half h, column i) receives tile[r0 + 4h + j]
// [c0 + i] (slots 0-3) and tile[r0 + 8 + 4h + j][c0 + i] (slots 4-7), j = 0..3,
// from two transposing reads in which source lane L of each 16-lane group
// points at row r0 + 4h + L/4 (+ 8), columns c0 + 16 (group & 1) + 4 (L % 4).
template <int W>
__device__ __forceinline__ bf16x8 tr_operand(const uint16_t* tile, int r0, int c0, int lane) {
    const int li = lane & 15, grp = lane >> 4, h = lane >> 5;
    const int col = c0 + 16 * (grp & 1) + 4 * (li & 3);
    const int row = r0 + 4 * h + (li >> 2);
    const v4s lo = tr_read(tile, toff<W>(row, col));
    const v4s hi = tr_read(tile, toff<W>(row + 8, col));
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

// This wave's share of the global->LDS copies of a 64-row tile of width W
// (16-byte chunks; chunk i * 256 + 64 wave + lane of the tile for copy i of a
// lane). LDS chunk (r, pos) receives global chunk (r, pos ^ swz(r)), which is the
// swizzled layout the reads expect. Rows at or past `rows` re-read row rows - 1:
// finite values, masked later.
template <int W>
struct TileCopy {
    static constexpr int CHUNKS = kT * W / 8;
    static constexpr int N = CHUNKS / kThreads;
    static_assert(CHUNKS % kThreads == 0, "tile chunks must spread evenly over the workgroup");
    // Copy i of a lane reads 256 chunks (4096 bytes) past copy i - 1: its row moves
    // by a multiple of 16 (W = 128) or 32 (W = 64) rows, which leaves swz unchanged.
    uint32_t off0;  // global byte offset (in the tile) of the lane's first chunk
    int row0;       // its tile row
    __device__ __forceinline__ TileCopy(int wave, int lane) {
        const int ci = wave * 64 + lane;
        const int r = ci / (W / 8), pos = ci % (W / 8);
        row0 = r;
        off0 = (uint32_t)((r * W + ((pos ^ swz<W>(r)) * 8)) * 2);
    }
    __device__ __forceinline__ void issue(const uint16_t* g, int first, int rows, uint16_t* tile, int wave) const {
        const char* t = (const char*)(g + (size_t)first * W);
        if (first + kT <= rows) {  // workgroup-uniform
#pragma unroll
            for (int i = 0; i < N; ++i)
                copy16_to_lds(t, off0 + i * kThreads * 16, tile + (i * kThreads + wave * 64) * 8);
            return;
        }
        const int last = rows - first - 1;
#pragma unroll
        for (int i = 0; i < N; ++i) {
            const int r = row0 + i * (kThreads * 8 / W);
            const uint32_t o = off0 + i * kThreads * 16;
            copy16_to_lds(t, r > last ? o - (r - last) * W * 2 : o, tile + (i * kThreads + wave * 64) * 8);
        }
    }
};

// A 16-wide contraction step of packed bf16 values from an accumulator: the
// registers 8 (q % 2) .. + 7 of block q / 2 (rows 16 q + 4h + j, 16 q + 8 + 4h + j).
__device__ __forceinline__ bf16x8 pack_step(const f32x16& x, int sub) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = pack_bf16(x[8 * sub + 2 * i], x[8 * sub + 2 * i + 1]);
    return __builtin_bit_cast(bf16x8, make_uint4(w[0], w[1], w[2], w[3]));
}

__device__ __forceinline__ float bf16_at(const uint4& w, int e) {
    const uint32_t x = e < 2 ? w.x : e < 4 ? w.y : e < 6 ? w.z : w.w;
    return (e & 1) ? bf16hi(x) : bf16lo(x);
}

// P = exp2(c S - lse2) and dS = P (dP - D) for the 16 rows 8 j + e (+ the lane's
// 4 half) of a 32-row block, in place of S and dP. lq, dq: the block's lse2 and D
// from the lane's first row. MASK: row u0 + 8 j + e counts only when it lies in
// [0, span) (the rows that see the lane's key, relative to the first of them).
template <bool MASK>
__device__ __forceinline__ void kv_probs(f32x16& s, f32x16& dp, const float* lq, const float* dq, float c, int u0,
                                         int span) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const float4 lj = *(const float4*)(lq + 8 * j);
        const float4 dj = *(const float4*)(dq + 8 * j);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int v = 4 * j + e;
            const float l = e == 0 ? lj.x : e == 1 ? lj.y : e == 2 ? lj.z : lj.w;
            const float dl = e == 0 ? dj.x : e == 1 ? dj.y : e == 2 ? dj.z : dj.w;
            float x = exp2_fast(fmaf(s[v], c, -l));
            if constexpr (MASK) x = (unsigned)(u0 + 8 * j + e) < (unsigned)span ? x : 0.f;
            s[v] = x;
            dp[v] = x * (dp[v] - dl);
        }
    }
}

// dS^T = P^T (dP^T - D) in place of S^T, P^T = exp2(c S^T - lse2), for the keys
// 8 (v/4) + v % 4 (+ the lane's 4 half) of a 32-key block. MASK: keys past
// `lim` (relative to the block's first key for this lane) weigh 0.
template <bool MASK>
__device__ __forceinline__ void q_dscores(f32x16& s, const f32x16& dp, float c, float lse2, float D, int lim) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        float pr = exp2_fast(fmaf(s[v], c, -lse2));
        if constexpr (MASK) pr = 8 * (v >> 2) + (v & 3) > lim ? 0.f : pr;
        s[v] = pr * (dp[v] - D);
    }
}

}  // namespace

// ------------------------------------------------------------------ dQ and D

template <int R, int DV>
struct alignas(16) DqSmem {
    uint16_t k[2][kT * R];
    uint16_t v[2][kT * DV];
};

template <int R, int DV>
__global__ __launch_bounds__(kThreads, 2) void bwd_dq_kernel(const PrefillBwdParams p, int n_groups) {
    constexpr int KSTEPS = R / 16, DSTEPS = DV / 16, RBLK = R / 32;
    __shared__ DqSmem<R, DV> sm;

    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = lane >> 5, col = lane & 31;

    // workgroup -> (KV sequence, 32 rows x HPW heads), XCD-aware, heaviest first
    const int HPW = gcd4(p.G);
    const int RB = 4 / HPW;
    const int BM = 32 * RB;
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
    const int qw0 = q0 + (wave / HPW) * 32;
    const int off = p.Sk - p.Sq;
    const int qrow = qw0 + col;
    const bool row_ok = qrow < p.Sq;
    const int qr = row_ok ? qrow : p.Sq - 1;

    const size_t rowq = (size_t)b * p.Hq + h;
    const uint16_t* qg = (const uint16_t*)p.q + rowq * p.Sq * R;
    const uint16_t* og = (const uint16_t*)p.o + rowq * p.Sq * DV;
    const uint16_t* dog = (const uint16_t*)p.dout + rowq * p.Sq * DV;
    const uint16_t* kg = (const uint16_t*)p.k + ((size_t)b * p.Hkv + g) * p.Sk * R;
    const uint16_t* vg = (const uint16_t*)p.v + ((size_t)b * p.Hkv + g) * p.Sk * DV;

    const TileCopy<R> kc(wave, lane);
    const TileCopy<DV> vc(wave, lane);
    kc.issue(kg, 0, p.Sk, sm.k[0], wave);
    vc.issue(vg, 0, p.Sk, sm.v[0], wave);

    // B operands: Q^T (dims 16m + 8 half .. + 7 of the lane's row) and dO^T; D from dO and O
    bf16x8 qreg[KSTEPS], dreg[DSTEPS];
#pragma unroll
    for (int m = 0; m < KSTEPS; ++m) qreg[m] = *(const bf16x8*)(qg + (size_t)qr * R + 16 * m + 8 * half);
    float D = 0.f;
#pragma unroll
    for (int m = 0; m < DSTEPS; ++m) {
        const uint4 dw = *(const uint4*)(dog + (size_t)qr * DV + 16 * m + 8 * half);
        const uint4 ow = *(const uint4*)(og + (size_t)qr * DV + 16 * m + 8 * half);
        dreg[m] = __builtin_bit_cast(bf16x8, dw);
#pragma unroll
        for (int e = 0; e < 8; ++e) D = fmaf(bf16_at(dw, e), bf16_at(ow, e), D);
    }
    D = xor32_sum(D);
    const float lse2 = p.lse[rowq * p.Sq + qr] * kLog2e;
    if (half == 0 && row_ok) {
        p.delta[rowq * p.Sq + qrow] = D;
        p.lse2[rowq * p.Sq + qrow] = lse2;
    }
    const float c = p.qscale;

    int key_end = p.Sk;
    if (p.causal) {
        const int last = q0 + BM + off;
        key_end = last < key_end ? last : key_end;
    }
    const int ntiles = (key_end + kT - 1) / kT;
    const int wave_last_key = p.causal ? qw0 + 31 + off : p.Sk - 1;
    const int lim = p.causal ? (qrow + off < p.Sk - 1 ? qrow + off : p.Sk - 1) : p.Sk - 1;

    f32x16 dq[RBLK];
#pragma unroll
    for (int rb = 0; rb < RBLK; ++rb)
#pragma unroll
        for (int v = 0; v < 16; ++v) dq[rb][v] = 0.f;

    wait_loads();
    // the same wait as a builtin, so that the compiler knows the row loads have
    // landed and adds no wait of its own inside the tile loop (vmcnt 0)
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();

    for (int t = 0; t < ntiles; ++t) {
        const int cur = t & 1;
        const int base = t * kT;
        if (t + 1 < ntiles) {
            kc.issue(kg, base + kT, p.Sk, sm.k[cur ^ 1], wave);
            vc.issue(vg, base + kT, p.Sk, sm.v[cur ^ 1], wave);
        }
        if (base <= wave_last_key) {
            const uint16_t* ks = sm.k[cur];
            const uint16_t* vs = sm.v[cur];
            const bool needs_mask = (p.causal && base + kT - 1 > qw0 + off) || base + kT > p.Sk;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                // S^T and dP^T of keys base + 32 kb + (8 (v/4) + 4 half + v % 4), query col
                f32x16 s, dp;
#pragma unroll
                for (int v = 0; v < 16; ++v) s[v] = dp[v] = 0.f;
#pragma unroll
                for (int m = 0; m < KSTEPS; ++m)
                    s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_operand<R>(ks, kb * 32 + col, 16 * m + 8 * half),
                                                                qreg[m], s, 0, 0, 0);
#pragma unroll
                for (int m = 0; m < DSTEPS; ++m)
                    dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        row_operand<DV>(vs, kb * 32 + col, 16 * m + 8 * half), dreg[m], dp, 0, 0, 0);
                // dS^T = P^T (dP^T - D), P^T = exp2(c S^T - log2-domain L); masked keys weigh 0
                if (needs_mask)
                    q_dscores<true>(s, dp, c, lse2, D, lim - (base + kb * 32 + 4 * half));
                else
                    q_dscores<false>(s, dp, c, lse2, D, 0);
                // dQ^T += K^T dS^T over the block's two 16-key steps
#pragma unroll
                for (int sub = 0; sub < 2; ++sub) {
                    const bf16x8 bop = pack_step(s, sub);
#pragma unroll
                    for (int rb = 0; rb < RBLK; ++rb)
                        dq[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            tr_operand<R>(ks, kb * 32 + 16 * sub, 32 * rb, lane), bop, dq[rb], 0, 0, 0);
                }
            }
        }
        if (t + 1 < ntiles) wait_loads();  // this wave's part of the next tile has landed
        __syncthreads();
    }

    // dQ rows: lane (half, col) holds dims 32 rb + 8 (v/4) + 4 half + v % 4 of row qrow
    if (row_ok) {
        uint16_t* dqrow = (uint16_t*)p.dq + (rowq * p.Sq + qrow) * R;
#pragma unroll
        for (int rb = 0; rb < RBLK; ++rb)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                uint2 w;
                w.x = pack_bf16(dq[rb][4 * j] * p.scale, dq[rb][4 * j + 1] * p.scale);
                w.y = pack_bf16(dq[rb][4 * j + 2] * p.scale, dq[rb][4 * j + 3] * p.scale);
                *(uint2*)(dqrow + rb * 32 + 8 * j + 4 * half) = w;
            }
    }
}

// ------------------------------------------------------------------ dK and dV

template <int R, int DV>
struct alignas(16) KvSmem {
    uint16_t q[2][kT * R];
    uint16_t d[2][kT * DV];
    float lse2[2][kT];  // log2-domain log-sum-exp of the tile's rows
    float dl[2][kT];    // D of the tile's rows
};

// Issue the copies of query tile `it` (head g G + it % G, rows from
// (t0 + n_rt - 1 - it / G) 64) into buffer `buf`: Q and dO rows by all waves, the rows'
// lse2 by wave 0 and D by wave 1 (one float per lane, rows clamped to Sq - 1).
template <int R, int DV>
__device__ __forceinline__ void issue_qtile(const PrefillBwdParams& p, KvSmem<R, DV>& sm, const TileCopy<R>& qc,
                                            const TileCopy<DV>& dc, int it, int buf, int b, int g, int t0,
                                            int n_rt, int wave, int lane) {
    const int hh = g * p.G + it % p.G;
    const int row0 = (t0 + n_rt - 1 - it / p.G) * kT;
    const size_t rowq = (size_t)b * p.Hq + hh;
    qc.issue((const uint16_t*)p.q + rowq * p.Sq * R, row0, p.Sq, sm.q[buf], wave);
    dc.issue((const uint16_t*)p.dout + rowq * p.Sq * DV, row0, p.Sq, sm.d[buf], wave);
    if (wave < 2) {
        int r = row0 + lane;
        r = r < p.Sq ? r : p.Sq - 1;
        const float* src = wave == 0 ? p.lse2 : p.delta;
        copy4_to_lds((const char*)(src + rowq * p.Sq), (uint32_t)r * 4u, wave == 0 ? sm.lse2[buf] : sm.dl[buf]);
    }
}

// Register budget: the dK and dV accumulators (r + d_v per lane) and the K and V
// rows fit two workgroups per CU while r + d_v < 192.
template <int R, int DV>
__global__ __launch_bounds__(kThreads, R + DV >= 192 ? 1 : 2) void bwd_dkdv_kernel(const PrefillBwdParams p,
                                                                                    int n_groups) {
    constexpr int KSTEPS = R / 16, DSTEPS = DV / 16, RBLK = R / 32, DBLK = DV / 32;
    constexpr int KB = 4 * 32;  // keys per workgroup
    __shared__ KvSmem<R, DV> sm;

    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = lane >> 5, col = lane & 31;

    // workgroup -> (KV sequence, 128 keys), XCD-aware, longest query range first
    const int nkb = (p.Sk + KB - 1) / KB;
    const int per_xcd = (n_groups + kXcds - 1) / kXcds;
    const int logical = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    if (logical >= n_groups) return;
    const int pair = logical / nkb, kbi = logical % nkb;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    const int k0g = kbi * KB;              // first key of the workgroup
    const int k0 = k0g + wave * 32;        // first key of the wave
    const int key = k0 + col;              // this lane's key (B-operand column)
    const bool key_ok = key < p.Sk;
    const int off = p.Sk - p.Sq;
    // rows that see this lane's key: [rmin, rmin + span)
    const int rmin = p.causal ? key - off : 0;
    const int span = key_ok ? p.Sq - rmin : 0;  // >= 1: key - off <= Sq - 1

    const size_t kvrow = (size_t)b * p.Hkv + g;
    const uint16_t* kg = (const uint16_t*)p.k + kvrow * p.Sk * R;
    const uint16_t* vg = (const uint16_t*)p.v + kvrow * p.Sk * DV;

    // query tiles that see any key of the workgroup
    int first_row = p.causal ? k0g - off : 0;
    first_row = first_row < 0 ? 0 : first_row;
    const int t0 = first_row / kT;
    const int nt = (p.Sq + kT - 1) / kT;
    const int n_rt = nt - t0;
    const int n_iter = n_rt * p.G;  // (tile, head) pairs, tiles descending, heads innermost

    const TileCopy<R> qc(wave, lane);
    const TileCopy<DV> dc(wave, lane);
    if (n_iter > 0) issue_qtile<R, DV>(p, sm, qc, dc, 0, 0, b, g, t0, n_rt, wave, lane);

    // B operands of S = Q K^T and dP = dO V^T: the lane's key row
    bf16x8 kreg[KSTEPS], vreg[DSTEPS];
#pragma unroll
    for (int m = 0; m < KSTEPS; ++m) {
        const uint4 w = key_ok ? *(const uint4*)(kg + (size_t)key * R + 16 * m + 8 * half) : make_uint4(0, 0, 0, 0);
        kreg[m] = __builtin_bit_cast(bf16x8, w);
    }
#pragma unroll
    for (int m = 0; m < DSTEPS; ++m) {
        const uint4 w = key_ok ? *(const uint4*)(vg + (size_t)key * DV + 16 * m + 8 * half) : make_uint4(0, 0, 0, 0);
        vreg[m] = __builtin_bit_cast(bf16x8, w);
    }
    const float c = p.qscale;

    f32x16 dva[DBLK], dka[RBLK];
#pragma unroll
    for (int d = 0; d < DBLK; ++d)
#pragma unroll
        for (int v = 0; v < 16; ++v) dva[d][v] = 0.f;
#pragma unroll
    for (int rb = 0; rb < RBLK; ++rb)
#pragma unroll
        for (int v = 0; v < 16; ++v) dka[rb][v] = 0.f;

    wait_loads();
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt 0, known to the compiler
    __syncthreads();

    for (int it = 0; it < n_iter; ++it) {
        const int cur = it & 1;
        const int i0 = (t0 + n_rt - 1 - it / p.G) * kT;  // first query row of the tile
        if (it + 1 < n_iter) issue_qtile<R, DV>(p, sm, qc, dc, it + 1, cur ^ 1, b, g, t0, n_rt, wave, lane);
        if (!(p.causal && i0 + kT - 1 + off < k0)) {  // some row of the tile sees the wave's keys
            const uint16_t* qs = sm.q[cur];
            const uint16_t* ds = sm.d[cur];
            const bool needs_mask = (p.causal && i0 + off < k0 + 31) || i0 + kT > p.Sq || k0 + 32 > p.Sk;
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                // S and dP of query rows i0 + 32 qb + (8 (v/4) + 4 half + v % 4), key col
                f32x16 s, dp;
#pragma unroll
                for (int v = 0; v < 16; ++v) s[v] = dp[v] = 0.f;
#pragma unroll
                for (int m = 0; m < KSTEPS; ++m)
                    s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_operand<R>(qs, qb * 32 + col, 16 * m + 8 * half),
                                                                kreg[m], s, 0, 0, 0);
#pragma unroll
                for (int m = 0; m < DSTEPS; ++m)
                    dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        row_operand<DV>(ds, qb * 32 + col, 16 * m + 8 * half), vreg[m], dp, 0, 0, 0);
                // P and dS = P (dP - D) replace S and dP in place; masked pairs weigh 0
                const float* lq = &sm.lse2[cur][qb * 32 + 4 * half];
                const float* dq = &sm.dl[cur][qb * 32 + 4 * half];
                if (needs_mask)
                    kv_probs<true>(s, dp, lq, dq, c, i0 + qb * 32 + 4 * half - rmin, span);
                else
                    kv_probs<false>(s, dp, lq, dq, c, 0, 0);
                // dV += P^T dO and dK += dS^T Q over the block's two 16-row steps
#pragma unroll
                for (int sub = 0; sub < 2; ++sub) {
                    const bf16x8 pa = pack_step(s, sub);
                    const bf16x8 sa = pack_step(dp, sub);
                    const int r0 = qb * 32 + 16 * sub;
#pragma unroll
                    for (int d = 0; d < DBLK; ++d)
                        dva[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pa, tr_operand<DV>(ds, r0, 32 * d, lane),
                                                                         dva[d], 0, 0, 0);
#pragma unroll
                    for (int rb = 0; rb < RBLK; ++rb)
                        dka[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(sa, tr_operand<R>(qs, r0, 32 * rb, lane),
                                                                          dka[rb], 0, 0, 0);
                }
            }
        }
        if (it + 1 < n_iter) wait_loads();  // this wave's part of the next tile has landed
        __syncthreads();
    }

    // dK, dV rows: lane (half, col) holds keys k0 + 8 (v/4) + 4 half + v % 4, column col of each block
    uint16_t* dkg = (uint16_t*)p.dk + kvrow * p.Sk * R;
    uint16_t* dvg = (uint16_t*)p.dv + kvrow * p.Sk * DV;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const int kk = k0 + 8 * (v >> 2) + 4 * half + (v & 3);
        if (kk >= p.Sk) continue;
#pragma unroll
        for (int rb = 0; rb < RBLK; ++rb)
            dkg[(size_t)kk * R + 32 * rb + col] = (uint16_t)(pack_bf16(dka[rb][v] * p.scale, 0.f) & 0xffffu);
#pragma unroll
        for (int d = 0; d < DBLK; ++d)
            dvg[(size_t)kk * DV + 32 * d + col] = (uint16_t)(pack_bf16(dva[d][v], 0.f) & 0xffffu);
    }
}

// ------------------------------------------------------------------ dispatch

template <int R, int DV>
static hipError_t run(const PrefillBwdParams& p, hipStream_t st) {
    const int HPW = gcd4(p.G);
    const int BM = 32 * (4 / HPW);
    const long nqb = (p.Sq + BM - 1) / BM;
    const long groups_q = nqb * p.Hkv * (p.G / HPW) * p.B;
    const long nkb = (p.Sk + 127) / 128;
    const long groups_k = nkb * p.Hkv * p.B;
    const long lq = (groups_q + kXcds - 1) / kXcds * kXcds, lk = (groups_k + kXcds - 1) / kXcds * kXcds;
    if (lq * kThreads > 0xffffffffL || lk * kThreads > 0xffffffffL) return hipErrorInvalidValue;
    if (lq > 0) {
        hipLaunchKernelGGL((bwd_dq_kernel<R, DV>), dim3((unsigned)lq), dim3(kThreads), 0, st, p, (int)groups_q);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (lk > 0) {
        hipLaunchKernelGGL((bwd_dkdv_kernel<R, DV>), dim3((unsigned)lk), dim3(kThreads), 0, st, p, (int)groups_k);
        return hipGetLastError();
    }
    return hipSuccess;
}

template <int R>
static hipError_t by_dv(const PrefillBwdParams& p, int DV, hipStream_t st) {
    if (DV == 64) return run<R, 64>(p, st);
    if (DV == 128) return run<R, 128>(p, st);
    return hipErrorInvalidValue;
}

tk_status launch_prefill_backward(const PrefillBwdParams& p, int R, int DV, hipStream_t st) {
    hipError_t e;
    switch (R) {
        case 32: e = by_dv<32>(p, DV, st); break;
        case 64: e = by_dv<64>(p, DV, st); break;
        case 128: e = by_dv<128>(p, DV, st); break;
        default: return TK_ERR_UNSUPPORTED;
    }
    if (e == hipErrorInvalidValue) return TK_ERR_UNSUPPORTED;
    return e == hipSuccess ? TK_OK : TK_ERR_HIP;
}

}  // namespace tk
