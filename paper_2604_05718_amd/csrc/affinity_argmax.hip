// Fused cosine affinity + self-masked row argmax (Eq. 1 and the nearest
// neighbour of Sec. 3.2) for gfx950.
//
// For image b with n tokens, every query i gets
//     nb[i] = argmax_{j != i, j < n} (x_i . x_j) * inv_j,   inv_j = 1 / max(||x_j||, 1e-12),
// with the lowest j kept among equal scores. Dividing the dot product by
// ||x_i|| as well would not move a row's argmax, so only the candidate norm is
// applied. The dot products come from MFMA on the stored values (bfloat16
// products are exact in float32, accumulation is float32); normalising first
// and rounding the unit vectors back to bfloat16 would cost about three
// decimal digits of the cosine, so the inputs are never rescaled.
//
// Tiling. A workgroup owns QT queries of one image and streams every
// candidate tile of CT tokens past them; the N x N affinity only ever lives
// in MFMA accumulators. Per candidate tile the K dimension (D) is staged
// through LDS in 128-byte chunks, double-buffered: the global loads of the
// next chunk are in flight while the current one feeds the MFMAs.
// In the 32x32 MFMA the candidate is the row operand and the query the column
// operand, so each lane's 16 accumulator values belong to ONE query and 16
// different candidates: the running (max, index) reduction is per lane, in
// registers, in ascending candidate order, and lanes/waves are merged
// lexicographically (larger score, then smaller index) only once at the end.
// The candidate norms are accumulated from the same register fragments that
// feed the MFMAs (one wave row per candidate slice), so X is read once per
// tile and no separate normalisation pass exists.
#include <hip/hip_ext.h>

#include <algorithm>
#include <vector>

#include "mpm_device.h"
#include "mpm_launch.h"

namespace mpm {
namespace {

template <class S>
struct Mfma;

template <>
struct Mfma<Bf16> {
    // 16 bytes per lane = 8 bfloat16 values along k: one 32x32x16 MFMA.
    static __device__ __forceinline__ void mma(f32x16& acc, u32x4 a, u32x4 b)
    {
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                      __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
    }
    // Sum of squares of the 8 values, accumulated into s: one v_dot2c_f32_bf16 per pair
    // (both squares and the running sum in one instruction, a quarter of the vector ALU
    // work of unpacking and two FMAs; its relative error on 768-value rows is at most
    // 1.6e-6 against float64, below the FMA chain's 3.5e-6). The words are copied to
    // scalars first: a bit cast of a subscripted element a[e] of the 4-word vector
    // compiled to four reads of its first word, and a cast of the whole fragment to 8
    // values cost 15-20 more VGPRs in the persistent kernels.
    static __device__ __forceinline__ float sumsq(u32x4 a, float s)
    {
        const uint32_t w0 = a.x, w1 = a.y, w2 = a.z, w3 = a.w;
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w0), __builtin_bit_cast(bf16x2, w0), s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w1), __builtin_bit_cast(bf16x2, w1), s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w2), __builtin_bit_cast(bf16x2, w2), s, false);
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w3), __builtin_bit_cast(bf16x2, w3), s, false);
        return s;
    }
};

template <>
struct Mfma<F32> {
    // 16 bytes per lane = 4 float32 values along k: four 32x32x2 MFMAs. Lane l
    // feeds k-slot l/32 of the instruction; both operands use the same
    // lane -> k assignment, so the sum runs over all 8 k of the 32-byte group.
    static __device__ __forceinline__ void mma(f32x16& acc, u32x4 a, u32x4 b)
    {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[e]), __uint_as_float(b[e]),
                                                       acc, 0, 0, 0);
    }
    static __device__ __forceinline__ float sumsq(u32x4 a, float s)
    {
#pragma unroll
        for (int e = 0; e < 4; ++e) s = fmaf(__uint_as_float(a[e]), __uint_as_float(a[e]), s);
        return s;
    }
};

constexpr int kXcds = 8;  // MI355X: workgroups are dealt round-robin to 8 XCDs, each with its own L2

// Workgroup barrier that waits only for this wave's LDS operations (not for
// outstanding global loads, which keep streaming into other LDS buffers).
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt unconstrained
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Register-staged variant (any 16-byte row size, float32 or bfloat16): a
// workgroup owns QT queries and loops over every candidate tile itself.
// WC x WQ waves; each wave computes MT x NT tiles of 32 candidates x 32 queries;
// CHUNK bytes of the K dimension are staged per LDS buffer.
//
// LOCAL: the locality constraint of Sec. 5 (candidates restricted to a window on the
// token grid; positions in `win`). A token's position is a raster index on a grid of
// win.grid_w columns (win.pos packed like x; null: the token's index in its image);
// j is a candidate of i when both lie within win.radius rows and columns of each
// other. Positions are non-decreasing in row along an image (raster order, which the
// left-to-right ids keep for merged tokens), so the candidates of a query block lie in
// a contiguous range of candidate tiles: only those are streamed, and every score is
// masked by the window test.
struct Window {
    const int32_t* pos;
    int grid_w, radius;
};

template <class S, int WC, int WQ, int MT, int NT, int CHUNK, bool LOCAL = false>
__global__ __launch_bounds__(WC * WQ * kWave) void affinity_argmax_kernel(
    const uint8_t* __restrict__ x, const int32_t* __restrict__ x_off, int B, int N, int D, int qblocks,
    int xcd_major, int T, float* __restrict__ pv, int32_t* __restrict__ pi, Window win)
{
    constexpr int THREADS = WC * WQ * kWave;
    constexpr int CT = WC * MT * 32;     // candidates per tile
    constexpr int QT = WQ * NT * 32;     // queries per workgroup
    constexpr int STRIDE = CHUNK + 16;   // padded LDS row pitch (bytes)
    constexpr int VPR = CHUNK / 16;      // 16-byte vectors per row per stage
    constexpr int CLOADS = CT * VPR / THREADS;
    constexpr int QLOADS = QT * VPR / THREADS;
    static_assert(CT * VPR % THREADS == 0 && QT * VPR % THREADS == 0, "tile/thread mismatch");

    __shared__ __attribute__((aligned(16))) uint8_t lds_c[2][CT * STRIDE];
    __shared__ __attribute__((aligned(16))) uint8_t lds_q[2][QT * STRIDE];
    __shared__ __attribute__((aligned(16))) float inv_c[2][CT];
    __shared__ float red_v[WC][QT];
    __shared__ int32_t red_i[WC][QT];
    __shared__ int16_t cand_rc[LOCAL ? 2 : 1][LOCAL ? 2 * CT : 1];  // grid row and column per candidate

    // Workgroup -> (image, query block). With xcd_major, consecutive ids that the
    // hardware sends to the same XCD walk through the query blocks of one image
    // before the next, so an image's candidate tiles are re-read from that XCD's L2.
    int b, qb;
    if (xcd_major) {
        const int xcd = blockIdx.x % kXcds;
        const int slot = blockIdx.x / kXcds;
        b = xcd + kXcds * (slot / qblocks);
        qb = slot % qblocks;
    } else {
        b = blockIdx.x / qblocks;
        qb = blockIdx.x % qblocks;
    }
    if (b >= B) return;
    const int qbase = qb * QT;
    const int row0 = x_off ? x_off[b] : b * N;
    const int n = x_off ? x_off[b + 1] - row0 : N;
    if (qbase >= n) return;  // uniform over the workgroup, before any barrier

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);  // wave-uniform: scalar registers and branches
    const int wc = wave % WC;
    const int wq = wave / WC;
    const int lrow = lane & 31;   // operand row inside a 32-row MFMA tile
    const int khalf = lane >> 5;  // which 16-byte half of a 32-byte k group

    const long rowbytes = (long)D * S::kBytes;
    const uint8_t* ximg = x + (long)row0 * rowbytes;
    const int nchunks = (int)((rowbytes + CHUNK - 1) / CHUNK);
    const int ntiles = (n + CT - 1) / CT;
    // Candidate tiles [t_lo, t_hi] (all of them without the locality constraint).
    int t_lo = 0, t_hi = ntiles - 1;
    auto grid_pos = [&](int i) { return win.pos ? win.pos[row0 + i] : i; };
    if (LOCAL) {
        const int r_first = grid_pos(qbase) / win.grid_w;
        const int r_last = grid_pos(min(qbase + QT, n) - 1) / win.grid_w;
        while (t_lo < ntiles - 1 && grid_pos(min((t_lo + 1) * CT, n) - 1) / win.grid_w < r_first - win.radius) ++t_lo;
        while (t_hi > t_lo && grid_pos(t_hi * CT) / win.grid_w > r_last + win.radius) --t_hi;
    }
    const int total = (t_hi - t_lo + 1) * nchunks;

    u32x4 pc[CLOADS];
    u32x4 pq[QLOADS];
    const u32x4 zero = {0u, 0u, 0u, 0u};

    auto gload = [&](int step) {
        const int tile = t_lo + step / nchunks;
        const long kb = (long)(step - (tile - t_lo) * nchunks) * CHUNK;
#pragma unroll
        for (int u = 0; u < CLOADS; ++u) {
            const int slot = tid + u * THREADS;
            const int r = slot / VPR;
            const long kk = kb + (slot % VPR) * 16;
            const int row = tile * CT + r;
            pc[u] = (row < n && kk < rowbytes) ? load16(ximg + row * rowbytes + kk) : zero;
        }
#pragma unroll
        for (int u = 0; u < QLOADS; ++u) {
            const int slot = tid + u * THREADS;
            const int r = slot / VPR;
            const long kk = kb + (slot % VPR) * 16;
            const int row = qbase + r;
            pq[u] = (row < n && kk < rowbytes) ? load16(ximg + row * rowbytes + kk) : zero;
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int u = 0; u < CLOADS; ++u) {
            const int slot = tid + u * THREADS;
            store16(&lds_c[buf][(slot / VPR) * STRIDE + (slot % VPR) * 16], pc[u]);
        }
#pragma unroll
        for (int u = 0; u < QLOADS; ++u) {
            const int slot = tid + u * THREADS;
            store16(&lds_q[buf][(slot / VPR) * STRIDE + (slot % VPR) * 16], pq[u]);
        }
    };

    f32x16 acc[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x16{};
    float ss[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) ss[mt] = 0.0f;
    float bv[NT];
    int32_t bi[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        bv[nt] = -__builtin_inff();
        bi[nt] = -1;
    }

    gload(0);
    lstore(0);
    __syncthreads();

    for (int step = 0; step < total; ++step) {
        const int buf = step & 1;
        if (step + 1 < total) gload(step + 1);

        const uint8_t* lc = lds_c[buf] + (wc * MT * 32 + lrow) * STRIDE + khalf * 16;
        const uint8_t* lq = lds_q[buf] + (wq * NT * 32 + lrow) * STRIDE + khalf * 16;
#pragma unroll
        for (int g = 0; g < CHUNK / 32; ++g) {
            u32x4 a[MT], q[NT];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                a[mt] = *reinterpret_cast<const u32x4*>(lc + mt * 32 * STRIDE + g * 32);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                q[nt] = *reinterpret_cast<const u32x4*>(lq + nt * 32 * STRIDE + g * 32);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) Mfma<S>::mma(acc[mt][nt], a[mt], q[nt]);
            // Candidate norms: m-tile mt is summed by the wave with wq == mt % WQ only.
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                if (mt % WQ == wq) ss[mt] = Mfma<S>::sumsq(a[mt], ss[mt]);
        }

        const int tile = t_lo + step / nchunks;
        const bool tile_end = (step - (tile - t_lo) * nchunks) == nchunks - 1;
        if (tile_end) {
            if constexpr (LOCAL) {
                // Grid row and column of each candidate of the tile (past the image: masked anyway).
                for (int jl = tid; jl < CT; jl += THREADS) {
                    const int j = tile * CT + jl;
                    const int p = j < n ? grid_pos(j) : 0;
                    cand_rc[tile & 1][2 * jl] = (int16_t)(p / win.grid_w);
                    cand_rc[tile & 1][2 * jl + 1] = (int16_t)(p % win.grid_w);
                }
            }
            // Lanes l and l+32 hold the two k halves of candidate row lrow.
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                if (mt % WQ != wq) continue;
                const float t = ss[mt] + __shfl_xor(ss[mt], 32);
                ss[mt] = 0.0f;
                if (khalf == 0) inv_c[tile & 1][wc * MT * 32 + mt * 32 + lrow] = 1.0f / fmaxf(sqrtf(t), 1e-12f);
            }
        }
        if (step + 1 < total) lstore(buf ^ 1);
        __syncthreads();

        if (tile_end) {
            // Epilogue: scale by the candidate's inverse norm, mask, running argmax.
            const int cb = tile * CT;
            const float* iv = inv_c[tile & 1];
            const bool need_mask = LOCAL || (cb + CT > n) || (cb < qbase + QT && qbase < cb + CT);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const int qi = qbase + wq * NT * 32 + nt * 32 + lrow;
                int q_r = 0, q_c = 0;  // this lane's query cell (locality constraint)
                if constexpr (LOCAL) {
                    const int p = qi < n ? grid_pos(qi) : 0;
                    q_r = p / win.grid_w;
                    q_c = p % win.grid_w;
                }
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        // Accumulator element 4g+e of this lane is candidate row 8g + 4*khalf + e.
                        const int jl = wc * MT * 32 + mt * 32 + 8 * g + 4 * khalf;
                        const f32x4 ivv = *reinterpret_cast<const f32x4*>(&iv[jl]);
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float s = acc[mt][nt][4 * g + e] * ivv[e];
                            const int j = cb + jl + e;
                            bool ok = !need_mask || (j < n && j != qi);
                            if constexpr (LOCAL) {
                                const int dr = cand_rc[tile & 1][2 * (jl + e)] - q_r;
                                const int dc = cand_rc[tile & 1][2 * (jl + e) + 1] - q_c;
                                ok = ok && dr <= win.radius && -dr <= win.radius && dc <= win.radius &&
                                     -dc <= win.radius;
                            }
                            if (ok && s > bv[nt]) {
                                bv[nt] = s;
                                bi[nt] = j;
                            }
                        }
                    }
                    acc[mt][nt] = f32x16{};
                }
            }
        }
    }

    // Merge the two lane halves (same query, interleaved candidate rows), then
    // the WC candidate waves, lexicographically: larger score, then smaller index.
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        float v = bv[nt];
        int32_t i = bi[nt];
        const float ov = __shfl_xor(v, 32);
        const int32_t oi = __shfl_xor(i, 32);
        if (ov > v || (ov == v && (uint32_t)oi < (uint32_t)i)) {
            v = ov;
            i = oi;
        }
        if (khalf == 0) {
            const int ql = wq * NT * 32 + nt * 32 + lrow;
            red_v[wc][ql] = v;
            red_i[wc][ql] = i;
        }
    }
    __syncthreads();
    for (int ql = tid; ql < QT; ql += THREADS) {
        const int qi = qbase + ql;
        if (qi >= n) continue;
        float v = red_v[0][ql];
        int32_t i = red_i[0][ql];
#pragma unroll
        for (int w = 1; w < WC; ++w) {
            const float ov = red_v[w][ql];
            const int32_t oi = red_i[w][ql];
            if (ov > v || (ov == v && (uint32_t)oi < (uint32_t)i)) {
                v = ov;
                i = oi;
            }
        }
        // This kernel covers every candidate itself: one partial, in tile slot 0.
        pv[(long)b * T * N + qi] = v;
        pi[(long)b * T * N + qi] = i;
    }
}

// Lane exchanges for the reverse-direction argmax of the symmetric schedule.
// Each DPP pattern used is an involution on the lanes of a 16-lane row.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ int32_t dpp_i(int32_t x)
{
    return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, false);
}
// (v, i) = the lexicographic maximum of (av, ai) and (bv, bi): larger score, then
// smaller index (as unsigned, so -1 loses every tie). Branch-free.
__device__ __forceinline__ void merge_pair(float& v, int32_t& i, float av, int32_t ai, float bv, int32_t bi)
{
    const bool c = (bv > av) | ((bv == av) & ((uint32_t)bi < (uint32_t)ai));
    v = c ? bv : av;
    i = c ? bi : ai;
}
// One reduce-scatter step over the H slot pairs (k, k+H): the partner lane (DPP
// pattern CTRL) keeps the other half. Lanes with `upper` keep slots k+H, the others
// slots k; each kept slot is merged with the partner's copy of it into slot k.
template <int CTRL, int H>
__device__ __forceinline__ void exchange_half(float* v, int32_t* ix, int upper)
{
#pragma unroll
    for (int k = 0; k < H; ++k) {
        const float kv = upper ? v[k + H] : v[k];
        const int32_t ki = upper ? ix[k + H] : ix[k];
        const float sv = upper ? v[k] : v[k + H];
        const int32_t si = upper ? ix[k] : ix[k + H];
        merge_pair(v[k], ix[k], kv, ki, dpp_f<CTRL>(sv), dpp_i<CTRL>(si));
    }
}

// Persistent variant for rows (bfloat16 or float32) that are a whole number of
// CB-byte chunks; everything below is laid out in bytes, and Mfma<S> consumes
// the same 16-byte fragments for either type. Work item = (image, query block of QT, candidate tile of CT); an item
// streams its two operand blocks through a STAGES-deep ring of LDS buffers
// filled by direct global->LDS loads (global_load_lds_dwordx4), runs the K loop
// on MFMA, then reduces its tile to one (score, index) partial per query.
//
// Scheduling for the 8 per-XCD L2 caches: workgroups are dealt round-robin to
// the XCDs, so workgroup w serves XCD group w % xcds; a group owns the images
// b = group + xcds * i and its `slots` workgroups take the group's items in
// order (item k goes to slot k % slots). All items of an image therefore run at
// the same time on one XCD, in lockstep over K, and each 256-row block is
// fetched from HBM once and re-read from that XCD's L2 by the other items that
// use it, instead of being refetched once per candidate tile.
//
// Pipeline. The chunks of all the workgroup's items form one stream. With
// STAGES >= 3, before chunk c is consumed this wave's loads of chunks up to c+1
// have landed and a barrier makes every wave's loads visible and retires the
// ring slot of chunk c-1, which is then refilled with chunk c+STAGES-1. Within a
// chunk the MFMA fragments are double-buffered: the fragments of the next
// k-group (for the last k-group: of the next chunk, already visible) are
// requested before the current k-group's MFMAs issue, so LDS latency hides
// behind the matrix cores. With STAGES == 2 (128-byte chunks: two stages fill
// 128 KB of LDS) the barrier before chunk c makes chunk c visible and retires
// chunk c-1's slot; chunk c's first fragments are requested, then chunk c+1's
// loads into the retired slot, so loads run one chunk ahead. Against 64-byte
// chunks in four stages this halves the barriers and the load instructions per
// byte, and each load instruction reads whole 128-byte lines.
// The global->LDS loads are written as assembly: the compiler cannot tell which
// ring slot they fill and would otherwise wait for all of them before every LDS
// read; their completion is waited for explicitly (vmcnt) instead.
//
// LDS layout of one stage: CB bytes of K per row (CB = 64 or 128), rows of an
// operand stored one after the other, with the CB/16 16-byte columns of a row
// permuted by an XOR swizzle: column c of row r sits in slot c ^ swz(r), with
//   CB = 128: swz(r) = ((r % 8) / 2) | (((r / 8) % 2) << 2),
//   CB =  64: swz(r) = (r / 4) % 4.
// One load instruction fills 1 KB = 1024/CB consecutive rows: lane l reads 16
// bytes of row l / (CB/16) (the lanes of a row cover its CB contiguous bytes of
// global memory) and lands at 16*l. An MFMA fragment read (one 16-byte column
// of 32 consecutive rows per lane half) then touches 16 distinct 16-byte bank
// groups in every 16-lane group, so it is free of bank conflicts on the
// 64-bank LDS. Load groups are dealt to the waves round-robin.
// Rows past the image are clamped to its last row (their scores are masked).
//
// Symmetric schedule (SYM). S = X X^T of an image is symmetric (Eq. 1), so only
// the blocks with query block <= candidate tile are computed: nb(nb+1)/2 items
// per image instead of nb^2. An off-diagonal item also yields the reverse
// direction: each candidate row j of the tile gets its best query q of the block,
// scored (x_j . x_q) * inv_q from the same accumulators, and writes the partial of
// row j for tile slot "query block". Every (row, slot) partial is still written
// exactly once, so the reduction over slots is unchanged. The products and sums
// are the same as in the item that would compute block (j's tile, q's block)
// directly, so the partials are bit-identical to the full schedule's. Items are
// taken image by image, the blocks of an image row by row, so all the items of
// an image still run together on one XCD and share its L2.
// Diagonal blocks taken out of a group's symmetric-schedule order (see HALVES below): with
// `whole` items on `slots` workgroups the last round holds m = whole mod slots items; when
// 0 < 2m <= slots and the group has at least m diagonal blocks, m of them are deferred.
__host__ __device__ inline int deferred_diagonals(int nimg, int nb, int slots)
{
    const int whole = nimg * (nb * (nb + 1) / 2);
    const int m = whole % slots;
    return (m > 0 && 2 * m <= slots && m <= nimg * nb) ? m : 0;
}

// HALVES: the second launch of a symmetric schedule on the two-stage ring. The first
// launch (SYM) leaves out the last deferred_diagonals() diagonal blocks of its XCD group
// (all of the last images', then the last ones of the image before), so that its slots
// take whole rounds; this launch runs each deferred block as two items of the block's
// 256 candidates and one half of its queries (QT = CT/2). A diagonal block needs no
// reverse direction, so the two halves write disjoint query partials, and each score
// comes from the same MFMA sequence as in a whole block.
//
// LOCAL: the locality constraint of Sec. 5 on the full schedule. A work item is a query
// block with every candidate tile its window band reaches ([tlo, thi], found from the
// positions at the block and tile boundaries, as in the register-staged kernel); the item
// runs its tiles one after the other through the same ring (one K loop per tile), keeps
// each query's running best across them in registers, masks every score by the window
// test, and writes one partial per query (tile slot 0, tile width N). Positions (win.pos,
// null: the token's index) are fetched per tile while its K loop runs, as given norms are.
//
// GIVEN (bfloat16 rows only): xinv holds the inverse row norms 1 / max(||x_j||, 1e-12),
// one float per row packed like x, which the kernel then takes instead of summing them
// from the fragments in the K loop (vector ALU work in the K loop adds to its time about
// one for one). Otherwise xinv is unused and every k-group's norm sums run without a
// branch; each case is its own build.
template <class S, int WC, int WQ, int MT, int NT, int CB, int STAGES, bool SYM, bool HALVES = false,
          bool LOCAL = false, bool GIVEN = false>
__global__ __launch_bounds__(WC * WQ * kWave, 2) void affinity_partial_kernel(  // 2 waves per SIMD
    const uint8_t* __restrict__ x, const int32_t* __restrict__ x_off, int B, int N, int D, int T, int xcds,
    int slots, float* __restrict__ pv, int32_t* __restrict__ pi, const float* __restrict__ xinv, Window win)
{
    constexpr int THREADS = WC * WQ * kWave;
    constexpr int WAVES = WC * WQ;
    constexpr int CT = WC * MT * 32;
    constexpr int QT = WQ * NT * 32;
    static_assert(CB == 64 || CB == 128, "swizzled layouts exist for 64- and 128-byte row chunks");
    constexpr int NS = CB / 16;                       // 16-byte slots per row
    constexpr int RPI = 64 / NS;                      // rows per load instruction (1 KB)
    // Rows a stage holds: the candidate tile, then the query block (none for a half item,
    // whose queries are rows of its own candidate tile).
    constexpr int QROWS = HALVES ? 0 : QT;
    constexpr int GROUPS = (CT + QROWS) / RPI;        // load instructions per stage
    constexpr int LOADS = GROUPS / WAVES;             // ... per wave
    constexpr int STAGE_BYTES = (CT + QROWS) * CB;
    constexpr int KG = CB / 32;                       // 32-byte k-groups (one MFMA k-step each) per chunk
    static_assert(GROUPS % WAVES == 0 && CT % RPI == 0 && CT % 32 == 0 && QT % 32 == 0, "stage/wave mismatch");
    static_assert(STAGES >= 2 && (STAGES - 2) * LOADS < 64, "pipeline depth / vmcnt range");
    static_assert(KG % 2 == 0, "the fragment double buffer alternates over an even number of k-groups");

    __shared__ __attribute__((aligned(1024))) uint8_t lds[STAGES * STAGE_BYTES];
    __shared__ __attribute__((aligned(16))) float inv_c[CT];
    __shared__ float red_v[WC][QT];
    __shared__ int32_t red_i[WC][QT];
    __shared__ __attribute__((aligned(16))) float inv_q[SYM ? QT : 1];
    __shared__ float red_cv[SYM ? WQ : 1][SYM ? CT : 1];
    __shared__ int32_t red_ci[SYM ? WQ : 1][SYM ? CT : 1];
    // LOCAL: grid row [0] and column [1] of the item's candidates (0 .. CT-1) and queries (CT ..).
    __shared__ __attribute__((aligned(16))) int32_t win_rc[2][LOCAL ? CT + QT : 1];
    static_assert(!LOCAL || (!HALVES && QT == CT && CT + QT <= WC * WQ * kWave),
                  "window items: square blocks, one position per thread");
    static_assert(!SYM || QT == CT, "the symmetric schedule pairs equal blocks");
    static_assert(CT + (SYM ? QT : 0) <= THREADS, "one given inverse norm per thread and item");
    static_assert(!GIVEN || S::kBytes == 2, "given norms: bfloat16 rows");
    constexpr bool given = GIVEN;

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);  // wave-uniform: scalar registers and branches
    const int wc = wave % WC;
    const int wq = wave / WC;
    const int lrow = lane & 31;
    const int khalf = lane >> 5;

    const int group = blockIdx.x % xcds;
    const int slot = blockIdx.x / xcds;
    const int nqb = (N + QT - 1) / QT;
    const int nct = (N + CT - 1) / CT;  // candidate tiles per image (T, the slot stride, may be larger)
    const int per_img = LOCAL ? nqb : (SYM ? nqb * (nqb + 1) / 2 : nqb * nct);
    const int nimg = (B - group + xcds - 1) / xcds;
    static_assert(!HALVES || (!SYM && 2 * QT == CT), "half items: forward only, half a block of queries");
    constexpr bool SPLIT = SYM && STAGES == 2 && !LOCAL;  // the layouts the second launch exists for
    const int ndef = (SPLIT || HALVES) ? deferred_diagonals(nimg, nct, slots) : 0;
    const int dfull = ndef / nct, dpart = ndef % nct;
    const int dimg = nimg - dfull - 1;                        // the image with dpart deferred
    const int upto_dimg = (dimg + 1) * per_img - dpart;       // first-launch items of images 0..dimg
    const int nitems = HALVES ? 2 * ndef : nimg * per_img - ndef;
    const long rowbytes = (long)D * S::kBytes;
    const int nchunks = (int)(rowbytes / CB);

    // Item cursor; all fields are uniform over the workgroup.
    struct Item {
        int k, b, qbase, cbase, n, row0;
        int tlo, thi;  // LOCAL: the item's band of candidate tiles (cbase walks up to thi)
    };
    auto find = [&](int k) {
        Item it;
        for (; k < nitems; k += slots) {
            int ib, qbase, t;
            if (HALVES) {  // deferred diagonal e, query half k % 2
                const int e = k >> 1;
                int qb;
                if (e < dpart) {
                    ib = dimg;
                    qb = nct - dpart + e;
                } else {
                    ib = dimg + 1 + (e - dpart) / nct;
                    qb = (e - dpart) - (ib - dimg - 1) * nct;
                }
                t = qb;
                qbase = qb * CT + (k & 1) * QT;
            } else if (LOCAL) {  // query block qb of image ib; its band's first tile is found below
                ib = k / nqb;
                t = k - ib * nqb;
                qbase = t * QT;
            } else if (SYM) {  // blocks qb <= t of the upper triangle, row by row, minus deferred diagonals
                int w;
                if (k < upto_dimg) {
                    ib = k / per_img;
                    w = k - ib * per_img;
                } else {
                    const int rest = max(1, per_img - nqb);
                    ib = dimg + 1 + (k - upto_dimg) / rest;
                    w = (k - upto_dimg) - (ib - dimg - 1) * rest;
                }
                const int d = ib > dimg ? nqb : (ib == dimg ? dpart : 0);  // image ib's deferred diagonals
                int qb = 0;
                for (;;) {
                    const int len = nqb - qb - (qb >= nqb - d ? 1 : 0);
                    if (w < len) break;
                    w -= len;
                    ++qb;
                }
                t = qb + w + (qb >= nqb - d ? 1 : 0);
                qbase = qb * QT;
            } else {
                ib = k / per_img;
                const int w = k - ib * per_img;
                const int qb = w / nct;
                t = w - qb * nct;
                qbase = qb * QT;
            }
            const int b = group + xcds * ib;
            const int row0 = x_off ? x_off[b] : b * N;
            const int n = x_off ? x_off[b + 1] - row0 : N;
            if (qbase < n && t * CT < n) {
                it.k = k; it.b = b; it.qbase = qbase; it.cbase = t * CT; it.n = n; it.row0 = row0;
                it.tlo = t;
                it.thi = t;
                if constexpr (LOCAL) {
                    // Candidate tiles whose grid rows can meet the block's window rows.
                    auto grid_row = [&](int i) { return (win.pos ? win.pos[row0 + i] : i) / win.grid_w; };
                    const int r_first = grid_row(qbase), r_last = grid_row(min(qbase + QT, n) - 1);
                    int tlo = 0, thi = (n - 1) / CT;
                    while (tlo < thi && grid_row(min((tlo + 1) * CT, n) - 1) < r_first - win.radius) ++tlo;
                    while (thi > tlo && grid_row(thi * CT) > r_last + win.radius) --thi;
                    // The symmetric schedule starts at the block's own tile: the tiles before
                    // it reach this block through their own items' reverse direction.
                    it.cbase = (SYM ? t : tlo) * CT;
                    it.tlo = tlo;
                    it.thi = thi;
                }
                return it;
            }
        }
        it.k = nitems; it.b = 0; it.qbase = 0; it.cbase = 0; it.n = 1; it.row0 = 0; it.tlo = 0; it.thi = 0;
        return it;
    };
    // The work after `it`: its next band tile (LOCAL), else the slot's next item.
    auto next_of = [&](const Item& it) {
        if constexpr (LOCAL) {
            if (it.cbase < it.thi * CT) {
                Item nx = it;
                nx.cbase += CT;
                return nx;
            }
        }
        return find(it.k + slots);
    };

    // Swizzle of the 16-byte column slot for a row (see the layout note above).
    auto swz = [](int r) {
        return CB == 128 ? (((r & 7) >> 1) | (((r >> 3) & 1) << 2)) : ((r >> 2) & 3);
    };
    const int lrowi = lane / NS;                          // row inside a load group
    const int lslot = lane % NS;                          // column slot this lane fills
    // Load group u = wave + WAVES * i covers rows u*RPI .. u*RPI+RPI-1 of [cand; query].
    // Byte offsets (from the image's first row) of this lane's 16-byte pieces for
    // the issue cursor's item; they change per item, not per chunk.
    struct Offsets {
        uint32_t v[LOADS];
    };
    auto offsets_of = [&](const Item& it) {
        Offsets o;
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            const int u = wave + WAVES * i;
            const bool is_q = u * RPI >= CT;
            const int r = u * RPI - (is_q ? CT : 0) + lrowi;   // row inside its operand block
            int row = (is_q ? it.qbase : it.cbase) + r;
            row = row < it.n ? row : it.n - 1;
            o.v[i] = (uint32_t)row * (uint32_t)rowbytes + (uint32_t)((lslot ^ swz(r & 15)) << 4);
        }
        return o;
    };

    Item ii = find(slot);  // issue cursor
    if (ii.k >= nitems) return;  // no work for this slot (uniform over the workgroup)
    Offsets ioff = offsets_of(ii);
    int ichunk = 0;
    int issued = 0;
    // The loads of a chunk are issued one at a time between the MFMAs of the chunk before
    // (issue_part, from mma_issue). Issued together after the barrier, a chunk's loads filled
    // the load queue and the wave stalled at issue with its MFMAs waiting behind them.
    uint8_t* isb = lds;
    const uint8_t* ibase = x;
    bool iact = false;
    auto issue_begin = [&]() {
        iact = ii.k < nitems;
        isb = lds + (issued % STAGES) * STAGE_BYTES;
        ibase = x + (long)ii.row0 * rowbytes + (long)ichunk * CB;   // uniform
    };
    // Once the issue cursor is past its last item the loads go on, unconditionally (no branch
    // per load in the K loop): they re-read rows of the last item (valid addresses) into the
    // ring slot after the last chunk, which nothing reads any more.
    auto issue_part = [&](int i) {
        const uint32_t off = ioff.v[i];
        const uint32_t m0 =
            (uint32_t)(size_t)(__attribute__((address_space(3))) uint8_t*)(isb + (wave + WAVES * i) * RPI * CB);
        // The LDS destination goes in M0, which the instruction reads implicitly: an input
        // operand bound to M0, so the compiler sets it and knows the asm reads it.
        asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(ibase), "{m0}"(m0) : "memory");
    };
    auto issue_end = [&]() {
        if (!iact) return;
        ++issued;
        if (++ichunk == nchunks) {
            ichunk = 0;
            ii = next_of(ii);
            if (ii.k < nitems) ioff = offsets_of(ii);
        }
    };
    auto issue_next = [&]() {
        issue_begin();
#pragma unroll
        for (int i = 0; i < LOADS; ++i) issue_part(i);
        issue_end();
    };

    // Row lrow of every 32-row fragment has the same swizzle (32 is a multiple of 16).
    const int sw = swz(lrow & 15);
    const int lc_off = (wc * MT * 32 + lrow) * CB;
    // A half item's queries are rows qbase - cbase.. of its candidate tile. Its first value
    // comes from the issue cursor's first item, which is the compute cursor's first item
    // (the prologue of a deeper ring reads fragments before the compute cursor exists); a
    // slot runs at most one half item (2 * ndef <= slots), so the read-ahead of a next
    // chunk never crosses into another half item.
    int lq_off = (HALVES ? ii.qbase - ii.cbase : CT) * CB + (wq * NT * 32 + lrow) * CB;
    u32x4 fa0[MT], fq0[NT], fa1[MT], fq1[NT];
    auto read_frags = [&](u32x4 (&fa)[MT], u32x4 (&fq)[NT], int chunk, int g) {
        const uint8_t* sb = lds + (chunk % STAGES) * STAGE_BYTES;
        const int col = ((2 * g + khalf) ^ sw) << 4;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) fa[mt] = *reinterpret_cast<const u32x4*>(sb + lc_off + mt * 32 * CB + col);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) fq[nt] = *reinterpret_cast<const u32x4*>(sb + lq_off + nt * 32 * CB + col);
    };

    f32x16 acc[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x16{};
    // Norm sums (rows not given): wave (wc, wq) sums candidate m-tiles wq, wq + WQ, ... and,
    // in the symmetric schedule, query n-tiles wc, wc + WC, ... It reads those fragments from
    // LDS a second time, before each k-group's MFMAs (own_c / own_q: their offsets in a stage,
    // before the k column), and sums them after the MFMAs. Picking them out of its registers
    // by wave index instead took a branch per tile in the K loop, which cost 5-8% of the
    // launch. An index past the wave's tiles reads its last tile, whose sum is unused.
    constexpr int NSC = (MT + WQ - 1) / WQ;
    constexpr int NSQ = SYM ? (NT + WC - 1) / WC : 1;
    float ss[NSC], sq[NSQ];
    int own_c[NSC], own_q[NSQ];
#pragma unroll
    for (int j = 0; j < NSC; ++j) {
        ss[j] = 0.0f;
        own_c[j] = lc_off + min(wq + j * WQ, MT - 1) * 32 * CB;
    }
#pragma unroll
    for (int j = 0; j < NSQ; ++j) {
        sq[j] = 0.0f;
        own_q[j] = min(wc + j * WC, NT - 1) * 32 * CB;  // from lq_off
    }
    // One load part before every PSTEP-th MFMA of a chunk: spread over all of the chunk's MFMAs
    // with STAGES >= 3, over the first half with two stages (those loads must land before the
    // chunk ends).
    constexpr int PGROUPS = KG * MT * NT;  // MFMAs per chunk
    constexpr int PSPAN = STAGES >= 3 ? PGROUPS : PGROUPS / 2;
    static_assert(PSPAN >= 1, "load parts per MFMA");
    constexpr int PSTEP = PSPAN >= LOADS ? PSPAN / LOADS : 1;              // MFMAs between load slots
    constexpr int PPER = PSPAN >= LOADS ? 1 : (LOADS + PSPAN - 1) / PSPAN;  // loads per slot (small tiles)
    auto mma_issue = [&](const u32x4 (&fa)[MT], const u32x4 (&fq)[NT], int chunk, int g) {
        u32x4 oc[NSC], oq[NSQ];
        if constexpr (!given) {
            const uint8_t* sb = lds + (chunk % STAGES) * STAGE_BYTES;
            const int col = ((2 * g + khalf) ^ sw) << 4;
#pragma unroll
            for (int j = 0; j < NSC; ++j) oc[j] = *reinterpret_cast<const u32x4*>(sb + own_c[j] + col);
            if constexpr (SYM) {
#pragma unroll
                for (int j = 0; j < NSQ; ++j) oq[j] = *reinterpret_cast<const u32x4*>(sb + lq_off + own_q[j] + col);
            }
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const int p = (g * MT + mt) * NT + nt;
                if (p % PSTEP == 0) {
#pragma unroll
                    for (int q = 0; q < PPER; ++q)
                        if ((p / PSTEP) * PPER + q < LOADS) issue_part((p / PSTEP) * PPER + q);
                }
                Mfma<S>::mma(acc[mt][nt], fa[mt], fq[nt]);
            }
        }
        if constexpr (!given) {
#pragma unroll
            for (int j = 0; j < NSC; ++j) ss[j] = Mfma<S>::sumsq(oc[j], ss[j]);
            if constexpr (SYM) {
#pragma unroll
                for (int j = 0; j < NSQ; ++j) sq[j] = Mfma<S>::sumsq(oq[j], sq[j]);
            }
        }
    };
    // vmcnt(n) with expcnt and lgkmcnt unconstrained.
    constexpr int kWaitAhead = 0x0F70 | ((((STAGES - 2) * LOADS) & 15)) | ((((STAGES - 2) * LOADS) >> 4) << 14);

    // Prologue: STAGES-1 chunks requested; with STAGES >= 3 chunk 0 has also landed, is
    // visible and has its first fragments requested (with two stages the loop does that).
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s) issue_next();
    if constexpr (STAGES >= 3) {
        if (issued == STAGES - 1) __builtin_amdgcn_s_waitcnt(kWaitAhead);
        else __builtin_amdgcn_s_waitcnt(0x0F70);
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        read_frags(fa0, fq0, 0, 0);
    }

    Item ci = find(slot);  // compute cursor
    // With given norms, thread t fetches the inverse norm of candidate row t (t < CT) or
    // query row t - CT (symmetric schedule) of the compute cursor's item when the cursor
    // reaches it; the value is written to LDS at the item's end. Rows past the image are
    // clamped, as the loads are.
    float inv_pre = 0.0f;
    auto fetch_inv = [&](const Item& it) {
        if (given && it.k < nitems) {
            const int r = tid < CT ? it.cbase + tid : it.qbase + tid - CT;
            if (tid < CT || (SYM && tid < CT + QT)) inv_pre = xinv[it.row0 + min(r, it.n - 1)];
        }
    };
    // LOCAL: thread t fetches the grid position of candidate row t or query row t - CT of
    // the compute cursor's tile; it goes to win_rc at the tile's end.
    int pos_pre = 0;
    auto fetch_pos = [&](const Item& it) {
        if (LOCAL && it.k < nitems && tid < CT + QT) {
            const int r = min(tid < CT ? it.cbase + tid : it.qbase + tid - CT, it.n - 1);
            pos_pre = win.pos ? win.pos[it.row0 + r] : r;
        }
    };
    fetch_inv(ci);
    fetch_pos(ci);
    // LOCAL: each query's best so far over the item's earlier tiles (this lane's n-tiles).
    float bv_run[LOCAL ? NT : 1];
    int32_t bi_run[LOCAL ? NT : 1];
#pragma unroll
    for (int nt = 0; nt < (LOCAL ? NT : 1); ++nt) {
        bv_run[nt] = -__builtin_inff();
        bi_run[nt] = -1;
    }
    int cchunk = 0;
    int consumed = 0;
    while (ci.k < nitems) {
        if constexpr (STAGES >= 3) {
            // This wave's loads of chunks up to c+1 have landed (later ones may stay in flight) ...
            const int ahead = issued - consumed - 2;
            if (ahead >= STAGES - 2) __builtin_amdgcn_s_waitcnt(kWaitAhead);
            else if (STAGES > 3 && ahead == 1)
                __builtin_amdgcn_s_waitcnt(0x0F70 | (LOADS & 15) | ((LOADS >> 4) << 14));
            else __builtin_amdgcn_s_waitcnt(0x0F70);
            // ... every wave's are visible, and every wave is done with chunk c-1's slot.
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            issue_begin();
        } else {
            // Chunk c has landed for this wave; after the barrier for every wave, and every
            // wave is done with chunk c-1, whose slot then takes chunk c+1.
            __builtin_amdgcn_s_waitcnt(0x0F70);
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            read_frags(fa0, fq0, consumed, 0);
            issue_begin();
        }
#pragma unroll
        for (int g = 0; g < KG; ++g) {
            if (g + 1 < KG) {
                if ((g & 1) == 0) read_frags(fa1, fq1, consumed, g + 1);
                else read_frags(fa0, fq0, consumed, g + 1);
            } else if (STAGES >= 3 && issued > consumed + 1) {
                read_frags(fa0, fq0, consumed + 1, 0);
            }
            if ((g & 1) == 0) mma_issue(fa0, fq0, consumed, g);
            else mma_issue(fa1, fq1, consumed, g);
        }
        issue_end();
        ++consumed;
        if (++cchunk < nchunks) continue;

        // ---- end of an item: norms, scores, per-query partial argmax ----
        if (given) {
            if (tid < CT) inv_c[tid] = inv_pre;
            else if (SYM && tid < CT + QT) inv_q[SYM ? tid - CT : 0] = inv_pre;
        } else {
#pragma unroll
            for (int j = 0; j < NSC; ++j) {
                const int mt = wq + j * WQ;
                if (mt >= MT) break;
                const float t = ss[j] + __shfl_xor(ss[j], 32);  // lanes l, l+32: the two k halves
                if (khalf == 0) inv_c[wc * MT * 32 + mt * 32 + lrow] = 1.0f / fmaxf(sqrtf(t), 1e-12f);
            }
            if constexpr (SYM) {
#pragma unroll
                for (int j = 0; j < NSQ; ++j) {
                    const int nt = wc + j * WC;
                    if (nt >= NT) break;
                    const float t = sq[j] + __shfl_xor(sq[j], 32);
                    if (khalf == 0) inv_q[wq * NT * 32 + nt * 32 + lrow] = 1.0f / fmaxf(sqrtf(t), 1e-12f);
                }
            }
        }
#pragma unroll
        for (int j = 0; j < NSC; ++j) ss[j] = 0.0f;
#pragma unroll
        for (int j = 0; j < NSQ; ++j) sq[j] = 0.0f;
        if constexpr (LOCAL) {
            if (tid < CT + QT) {
                win_rc[0][tid] = pos_pre / win.grid_w;
                win_rc[1][tid] = pos_pre % win.grid_w;
            }
        }
        lds_barrier();
        const float* iv = inv_c;
        const int n = ci.n;
        const int cb = ci.cbase;
        // 32-row tiles of this wave that hold at least one token of the image (uniform);
        // the others are computed on clamped rows and skipped here.
        const int mt_lim = min(MT, max(0, (n - (cb + wc * MT * 32) + 31) / 32));
        const int nt_lim = min(NT, max(0, (n - (ci.qbase + wq * NT * 32) + 31) / 32));
        // Query blocks are aligned and no larger than candidate tiles, so a query's own
        // index is a candidate of this item only when its block lies inside the tile;
        // it then sits in candidate 32-row tile (qbase - cb)/32 + (query 32-row tile).
        static_assert(CT % QT == 0, "query blocks must nest in candidate tiles");
        const bool diag = ci.qbase >= cb && ci.qbase < cb + CT;
        const int self_tile0 = (ci.qbase - cb) / 32;
        // Accumulator element r = 4g+e of this lane is candidate row 8g + 4*khalf + e of
        // its 32-row tile, so rows ascend with r. Each 16-value group is reduced by a
        // tournament in which the left (lower) entry wins ties, then merged into the
        // running best in ascending tile order with a strict >: the lowest index
        // wins among equal scores, as in a left-to-right scan.
        float bv[NT];
        int32_t bi[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            bv[nt] = LOCAL ? bv_run[LOCAL ? nt : 0] : -__builtin_inff();
            bi[nt] = LOCAL ? bi_run[LOCAL ? nt : 0] : -1;
        }
        // LOCAL: this lane's query's grid row and column per n-tile; the window test is
        // |row_j - row_q| <= radius and |col_j - col_q| <= radius, as unsigned compares.
        int q_r[LOCAL ? NT : 1], q_c[LOCAL ? NT : 1];
        if constexpr (LOCAL) {
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                q_r[nt] = win_rc[0][CT + wq * NT * 32 + nt * 32 + lrow] - win.radius;
                q_c[nt] = win_rc[1][CT + wq * NT * 32 + nt * 32 + lrow] - win.radius;
            }
        }
        const uint32_t wspan = 2u * (uint32_t)win.radius;
        // This lane's own row inside a 32-row tile, as an accumulator element (if it holds it).
        const int self_r = (((lrow >> 2) & 1) == khalf) ? 4 * (lrow >> 3) + (lrow & 3) : -1;
        if constexpr (LOCAL && SYM) {
            // Both directions read the accumulators: pairs outside the window become -inf
            // there (the inverse norms that scale them are positive).
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int jl = wc * MT * 32 + mt * 32 + 8 * g + 4 * khalf;
                    const int4 cr = *reinterpret_cast<const int4*>(&win_rc[0][jl]);
                    const int4 cc = *reinterpret_cast<const int4*>(&win_rc[1][jl]);
                    const int crv[4] = {cr.x, cr.y, cr.z, cr.w}, ccv[4] = {cc.x, cc.y, cc.z, cc.w};
#pragma unroll
                    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const bool in = (uint32_t)(crv[e] - q_r[nt]) <= wspan && (uint32_t)(ccv[e] - q_c[nt]) <= wspan;
                            acc[mt][nt][4 * g + e] = in ? acc[mt][nt][4 * g + e] : -__builtin_inff();
                        }
                }
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            if (mt >= mt_lim) break;
            const int jt = cb + wc * MT * 32 + mt * 32 + 4 * khalf;  // candidate of r = 0
            f32x4 ivv[4];
#pragma unroll
            for (int g = 0; g < 4; ++g)
                ivv[g] = *reinterpret_cast<const f32x4*>(&iv[wc * MT * 32 + mt * 32 + 8 * g + 4 * khalf]);
            const bool partial = cb + wc * MT * 32 + mt * 32 + 32 > n;  // some rows of this tile are past the image
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                if (nt >= nt_lim) break;
                float sc[16];
#pragma unroll
                for (int g = 0; g < 4; ++g)
#pragma unroll
                    for (int e = 0; e < 4; ++e) sc[4 * g + e] = acc[mt][nt][4 * g + e] * ivv[g][e];
                if (partial) {
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        sc[r] = jt + 8 * (r >> 2) + (r & 3) < n ? sc[r] : -__builtin_inff();
                }
                if (diag && wc * MT + mt == self_tile0 + wq * NT + nt) {  // the tile holding each lane's own query
#pragma unroll
                    for (int r = 0; r < 16; ++r) sc[r] = r == self_r ? -__builtin_inff() : sc[r];
                }
                if constexpr (LOCAL && !SYM) {
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int jl = wc * MT * 32 + mt * 32 + 8 * g + 4 * khalf;
                        const int4 cr = *reinterpret_cast<const int4*>(&win_rc[0][jl]);
                        const int4 cc = *reinterpret_cast<const int4*>(&win_rc[1][jl]);
                        const int crv[4] = {cr.x, cr.y, cr.z, cr.w}, ccv[4] = {cc.x, cc.y, cc.z, cc.w};
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const bool in = (uint32_t)(crv[e] - q_r[nt]) <= wspan && (uint32_t)(ccv[e] - q_c[nt]) <= wspan;
                            sc[4 * g + e] = in ? sc[4 * g + e] : -__builtin_inff();
                        }
                    }
                }
                float v8[8];
                int r8[8];
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const bool c = sc[2 * k + 1] > sc[2 * k];
                    v8[k] = c ? sc[2 * k + 1] : sc[2 * k];
                    r8[k] = c ? 2 * k + 1 : 2 * k;
                }
                float v4[4];
                int r4[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const bool c = v8[2 * k + 1] > v8[2 * k];
                    v4[k] = c ? v8[2 * k + 1] : v8[2 * k];
                    r4[k] = c ? r8[2 * k + 1] : r8[2 * k];
                }
                const bool c0 = v4[1] > v4[0];
                const float v20 = c0 ? v4[1] : v4[0];
                const int r20 = c0 ? r4[1] : r4[0];
                const bool c1 = v4[3] > v4[2];
                const float v21 = c1 ? v4[3] : v4[2];
                const int r21 = c1 ? r4[3] : r4[2];
                const bool cf = v21 > v20;
                const float v1 = cf ? v21 : v20;
                int r1 = cf ? r21 : r20;
                // Materialise the winning index before the merge: otherwise the compiler moves
                // the index selection into a divergent branch per tile, which serialises the
                // tiles' tournaments (measured slower).
                asm volatile("" : "+v"(r1));
                const bool up = v1 > bv[nt];
                bv[nt] = up ? v1 : bv[nt];
                bi[nt] = up ? jt + r1 + 4 * (r1 >> 2) : bi[nt];  // row 8*(r/4) + r%4 of the tile
            }
        }
        // Reverse direction of an off-diagonal item (query block before the candidate
        // tile). A candidate row's queries of one n-tile sit in the 32 lanes of one lane
        // half (one per lane), so after an in-lane merge over the NT n-tiles the best of
        // each row is found by a reduce-scatter across the half: exchanges with lane
        // l^16, l^15, l^7, l^2 and l^1 (XOR masks spanning all five lane bits) each
        // halve the rows a lane carries, until lanes 2r and 2r+1 hold row r's best.
        // Merges are lexicographic (larger score, then smaller query), so the lowest
        // query wins ties, as in the forward direction.
        const bool rev = SYM && !diag;
        if (rev) {
            float ivq[NT];
            bool qok[NT];
            int32_t qidx[NT];
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const int ql = wq * NT * 32 + nt * 32 + lrow;
                ivq[nt] = inv_q[ql];
                qidx[nt] = ci.qbase + ql;
                qok[nt] = qidx[nt] < n;
            }
            const bool all_q = ci.qbase + (wq + 1) * NT * 32 <= n;  // every query of this wave is a token (uniform)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                if (mt >= mt_lim) break;
                // This lane's best query for each of its 16 accumulator rows (a strict >
                // keeps the lower n-tile, i.e. the lower query, on ties).
                float v[16];
                int32_t ix[16];
                if (all_q) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        v[r] = acc[mt][0][r] * ivq[0];
                        ix[r] = qidx[0];
#pragma unroll
                        for (int nt = 1; nt < NT; ++nt) {
                            const float s2 = acc[mt][nt][r] * ivq[nt];
                            const bool c = s2 > v[r];
                            v[r] = c ? s2 : v[r];
                            ix[r] = c ? qidx[nt] : ix[r];
                        }
                    }
                } else {
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        v[r] = qok[0] ? acc[mt][0][r] * ivq[0] : -__builtin_inff();
                        ix[r] = qidx[0];
#pragma unroll
                        for (int nt = 1; nt < NT; ++nt) {
                            const float s2 = qok[nt] ? acc[mt][nt][r] * ivq[nt] : -__builtin_inff();
                            const bool c = s2 > v[r];
                            v[r] = c ? s2 : v[r];
                            ix[r] = c ? qidx[nt] : ix[r];
                        }
                    }
                }
                // l^16 with v_permlane16_swap: slots k and k+8 of the two 16-lane rows of a
                // half trade places, and the lower row keeps rows k, the upper rows k+8.
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const auto sv = __builtin_amdgcn_permlane16_swap(__float_as_uint(v[k]), __float_as_uint(v[k + 8]),
                                                                     false, false);
                    const auto si = __builtin_amdgcn_permlane16_swap((uint32_t)ix[k], (uint32_t)ix[k + 8], false, false);
                    merge_pair(v[k], ix[k], __uint_as_float(sv[0]), (int32_t)si[0], __uint_as_float(sv[1]),
                               (int32_t)si[1]);
                }
                exchange_half<0x140, 4>(v, ix, (lane >> 3) & 1);  // l^15 (row mirror), split on lane bit 3
                exchange_half<0x141, 2>(v, ix, (lane >> 2) & 1);  // l^7 (half-row mirror), bit 2
                exchange_half<0x4E, 1>(v, ix, (lane >> 1) & 1);   // l^2 (quad permutation 2,3,0,1), bit 1
                merge_pair(v[0], ix[0], v[0], ix[0], dpp_f<0xB1>(v[0]), dpp_i<0xB1>(ix[0]));  // l^1 (1,0,3,2)
                // Lanes 2r, 2r+1 of half h: accumulator row r = candidate row 8(r/4) + 4h + r%4.
                if ((lane & 1) == 0) {
                    const int r = (lrow >> 1) & 15;
                    const int jl = wc * MT * 32 + mt * 32 + 8 * (r >> 2) + 4 * khalf + (r & 3);
                    red_cv[wq][jl] = v[0];
                    red_ci[wq][jl] = ix[0];
                }
            }
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x16{};  // the next item starts from zero
        // LOCAL: between the tiles of an item only the running best is kept; the lanes,
        // waves and the partial are merged and written after its last tile.
        bool item_end = true;
        if constexpr (LOCAL) {
            item_end = ci.cbase >= ci.thi * CT;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                bv_run[nt] = item_end ? -__builtin_inff() : bv[nt];
                bi_run[nt] = item_end ? -1 : bi[nt];
            }
        }
        if (item_end) {
            // Merge the two lane halves, then the WC candidate waves (larger score, then smaller index).
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                float v = bv[nt];
                int32_t i = bi[nt];
                const float ov = __shfl_xor(v, 32);
                const int32_t oi = __shfl_xor(i, 32);
                if (ov > v || (ov == v && (uint32_t)oi < (uint32_t)i)) {
                    v = ov;
                    i = oi;
                }
                if (khalf == 0) {
                    const int ql = wq * NT * 32 + nt * 32 + lrow;
                    red_v[wc][ql] = v;
                    red_i[wc][ql] = i;
                }
            }
        }
        if (item_end || rev) lds_barrier();  // uniform
        if (item_end) {
            // The query block's partial: tile slot t (LOCAL: slot 0, or the block's own slot
            // under the symmetric schedule, whose earlier slots take the reverse direction).
            const int t = LOCAL ? (SYM ? ci.qbase / QT : 0) : cb / CT;
            for (int ql = tid; ql < QT; ql += THREADS) {
                const int qi = ci.qbase + ql;
                if (qi >= n) continue;
                float v = red_v[0][ql];
                int32_t i = red_i[0][ql];
#pragma unroll
                for (int w = 1; w < WC; ++w) {
                    const float ov = red_v[w][ql];
                    const int32_t oi = red_i[w][ql];
                    if (ov > v || (ov == v && (uint32_t)oi < (uint32_t)i)) {
                        v = ov;
                        i = oi;
                    }
                }
                const long o = ((long)ci.b * T + t) * N + qi;
                pv[o] = v;
                pi[o] = i;
                if constexpr (LOCAL && SYM) {
                    // The slots no item writes for this block's rows: tiles before the band and
                    // after the block (the band relation is symmetric, so the items that write
                    // slot q for these rows are exactly the blocks q of the band before it).
                    const int nq = (n + QT - 1) / QT;
                    for (int q = 0; q < nq; ++q) {
                        if (q >= ci.tlo && q <= t) continue;
                        const long oq = ((long)ci.b * T + q) * N + qi;
                        pv[oq] = -__builtin_inff();
                        pi[oq] = -1;
                    }
                }
            }
        }
        if (rev) {
            // Candidate rows of the tile over the query block: tile slot qbase / QT of their partials.
            const int tq = ci.qbase / QT;
            for (int jl = tid; jl < CT; jl += THREADS) {
                const int j = cb + jl;
                if (j >= n) continue;
                float v = red_cv[0][jl];
                int32_t i = red_ci[0][jl];
#pragma unroll
                for (int w = 1; w < WQ; ++w) merge_pair(v, i, v, i, red_cv[w][jl], red_ci[w][jl]);
                // A row with no query of the block inside its window: -inf, and no index.
                if (LOCAL && v == -__builtin_inff()) i = -1;
                const long o = ((long)ci.b * T + tq) * N + j;
                pv[o] = v;
                pi[o] = i;
            }
        }
        cchunk = 0;
        ci = next_of(ci);
        fetch_inv(ci);
        fetch_pos(ci);
        if constexpr (HALVES) lq_off = (ci.qbase - ci.cbase + wq * NT * 32 + lrow) * CB;
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);  // the trailing loads land before the workgroup's LDS is released
}

// Persistent-kernel shape: 256 candidates x 256 queries on 8 waves, 128-byte K
// chunks in a 2-deep ring (or 64-byte chunks 4 deep; 128 KB of LDS either way),
// one workgroup per CU. The full
// schedule splits the tile over 2 candidate x 4 query waves (128 x 64 each); the
// symmetric one over 4 x 2 (64 x 128 each), so that its reverse direction merges 4
// queries inside each lane before the cross-lane steps and carries half as many
// rows through them.
constexpr int kPWC = 2, kPWQ = 4, kPMT = 4, kPNT = 2, kPCB = 64, kPWGS = 1;
// Rows that are a whole number of 128-byte chunks stream them through two stages;
// other multiples of 64 bytes use 64-byte chunks in four stages.
constexpr int kPCB2 = 128;
constexpr int kSWC = 4, kSWQ = 2, kSMT = 2, kSNT = 4;
constexpr int kPCT = kPWC * kPMT * 32;
// Small batches (few 256 x 256 blocks for the device's CUs) use 64 x 64 blocks on 4 waves
// of one 32 x 32 tile each, so a single image of 1024 tokens still spreads over 256 CUs.
constexpr int kTWC = 2, kTWQ = 2, kTMT = 1, kTNT = 1;
constexpr int kTCT = kTWC * kTMT * 32;
constexpr long kSmallItems = 32;  // batches with at most this many 256 x 256 blocks take them
static_assert(kTWQ * kTNT * 32 == kTCT && kPCT % kTCT == 0, "square small blocks that nest in the large ones");
static_assert(kSWC * kSMT * 32 == kPCT && kSWQ * kSNT * 32 == kPCT && kPWQ * kPNT * 32 == kPCT,
              "both schedules use 256 x 256 tiles, so their partials share one layout");

bool use_persistent(int D, int dt) { return ((long)D * (dt == kBf16 ? 2 : 4)) % kPCB == 0; }

}  // namespace

bool affinity_takes_norms(int D, int dt) { return dt == kBf16 && use_persistent(D, dt); }

namespace {

int device_cus()
{
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    return cus;
}

// Whether a symmetric launch on the two-stage ring defers diagonal blocks in any XCD group.
bool defers_diagonals(int B, int N, int xcds, int slots)
{
    const int nb = (N + kPCT - 1) / kPCT;
    for (int g = 0; g < xcds; ++g)
        if (deferred_diagonals((B - g + xcds - 1) / xcds, nb, slots) > 0) return true;
    return false;
}

template <class S, int WC, int WQ, int MT, int NT, bool SYM, bool LOCAL, bool GIVEN>
void launch_persistent_as(const void* x, const int32_t* x_off, const float* xinv, int B, int N, int D, int T, int xcds,
                       int groups, float* pv, int32_t* pi, hipStream_t stream, hipEvent_t start, hipEvent_t stop,
                       Window win = Window{nullptr, 1, 0})
{
    const uint8_t* xb = static_cast<const uint8_t*>(x);
    if (((long)D * S::kBytes) % kPCB2 == 0) {
        // The symmetric schedule's deferred diagonal blocks, as half blocks, in a second launch
        // (one item per slot); the timing events then span both.
        const bool halves = SYM && !LOCAL && defers_diagonals(B, N, xcds, groups / xcds);
        hipExtLaunchKernelGGL((affinity_partial_kernel<S, WC, WQ, MT, NT, kPCB2, 2, SYM, false, LOCAL, GIVEN>), dim3(groups),
                              dim3(WC * WQ * kWave), 0, stream, start, halves ? nullptr : stop, 0, xb, x_off, B, N,
                              D, T, xcds, groups / xcds, pv, pi, xinv, win);
        if constexpr (SYM) {
            if (halves)
                hipExtLaunchKernelGGL((affinity_partial_kernel<S, WC, WQ, MT, NT / 2, kPCB2, 2, false, true, false, GIVEN>),
                                      dim3(groups), dim3(WC * WQ * kWave), 0, stream, nullptr, stop, 0, xb, x_off, B,
                                      N, D, T, xcds, groups / xcds, pv, pi, xinv, win);
        }
    } else
        hipExtLaunchKernelGGL((affinity_partial_kernel<S, WC, WQ, MT, NT, kPCB, 4, SYM, false, LOCAL, GIVEN>), dim3(groups),
                              dim3(WC * WQ * kWave), 0, stream, start, stop, 0, xb, x_off, B, N, D, T, xcds,
                              groups / xcds, pv, pi, xinv, win);
}

// Given norms (bfloat16 only) and norms summed in the K loop are separate builds: with one
// build and a run-time flag, the flag's branch per k-group cost the summing launches 2-4%,
// and two builds alternating between insertions showed no instruction-cache penalty.
template <class S, int WC, int WQ, int MT, int NT, bool SYM, bool LOCAL = false>
void launch_persistent(const void* x, const int32_t* x_off, const float* xinv, int B, int N, int D, int T, int xcds,
                       int groups, float* pv, int32_t* pi, hipStream_t stream, hipEvent_t start, hipEvent_t stop,
                       Window win = Window{nullptr, 1, 0})
{
    if constexpr (S::kBytes == 2) {
        if (xinv != nullptr) {
            launch_persistent_as<S, WC, WQ, MT, NT, SYM, LOCAL, true>(x, x_off, xinv, B, N, D, T, xcds, groups, pv,
                                                                      pi, stream, start, stop, win);
            return;
        }
    }
    launch_persistent_as<S, WC, WQ, MT, NT, SYM, LOCAL, false>(x, x_off, nullptr, B, N, D, T, xcds, groups, pv, pi,
                                                               stream, start, stop, win);
}

template <class S, int WC, int WQ, int MT, int NT, int CHUNK, bool LOCAL = false>
hipError_t launch_staged(const void* x, const int32_t* x_off, int B, int N, int D, int T, float* pv, int32_t* pi,
                         hipStream_t stream, hipEvent_t start, hipEvent_t stop, Window win = Window{nullptr, 1, 0})
{
    constexpr int QT = WQ * NT * 32;
    const int qblocks = (N + QT - 1) / QT;
    const int xcd_major = B >= kXcds ? 1 : 0;
    const long groups = xcd_major ? (long)kXcds * ((B + kXcds - 1) / kXcds) * qblocks : (long)B * qblocks;
    hipExtLaunchKernelGGL((affinity_argmax_kernel<S, WC, WQ, MT, NT, CHUNK, LOCAL>), dim3((unsigned)groups),
                          dim3(WC * WQ * kWave), 0, stream, start, stop, 0, static_cast<const uint8_t*>(x), x_off, B, N,
                          D, qblocks, xcd_major, T, pv, pi, win);
    return hipGetLastError();
}

}  // namespace

// Partial slots reserved per token: enough for the smallest block width any schedule uses.
int partial_tiles(int N) { return (N + kTCT - 1) / kTCT; }

bool valid_schedule(int schedule)
{
    return schedule == kScheduleAuto || schedule == kScheduleFull || schedule == kScheduleSymmetric ||
           schedule == kScheduleFull64;
}

namespace {

// Whether a persistent launch of this shape and requested schedule uses the 64 x 64
// blocks (no device query).
bool small_blocks(int B, int N, int schedule)
{
    if (schedule != kScheduleAuto) return schedule == kScheduleFull64;
    const long nqb = (N + kPCT - 1) / kPCT;
    return (long)B * nqb * nqb <= kSmallItems;
}

bool symmetric_schedule(int B, int N, int xcds, int slots, int schedule)
{
    if (schedule != kScheduleAuto) return schedule == kScheduleSymmetric;
    // Rounds of work items per workgroup slot under either schedule. An off-diagonal
    // item of the symmetric one costs about a fifth more (its reverse direction), so
    // it pays only when it saves more than that in rounds.
    const long nqb = (N + kPCT - 1) / kPCT;
    const long nimg = (B + xcds - 1) / xcds;
    const long full = (nimg * nqb * nqb + slots - 1) / slots;
    const long sym = (nimg * nqb * (nqb + 1) / 2 + slots - 1) / slots;
    return 5 * sym < 4 * full;
}

// The locality-constrained schedule's two block sizes: 256 x 256 blocks on 8 waves, one
// workgroup per CU (the dense symmetric shape), or 128 x 128 blocks on 4 waves of 64 x 64,
// two workgroups per CU. Smaller blocks cut a query block's window band more finely and
// give twice the items; each small block costs about 0.357 of a large one (a quarter of
// its matrix work at about 70% of its efficiency: half the flops per byte loaded).
constexpr int kLWC = 2, kLWQ = 2, kLMT = 2, kLNT = 2, kLWGS = 2;
constexpr int kLCT = kLWC * kLMT * 32;
static_assert(kLWQ * kLNT * 32 == kLCT && kPCT % kLCT == 0 && kLCT % kTCT == 0, "square small window blocks");
constexpr double kLSmallBlockCost = 0.357;

// Estimated duration (in large-block times) of a locality-constrained launch with ts x ts
// blocks, on a full raster grid (positions = token indices): per XCD group, the blocks of
// its images are dealt to the slots in order, each costing the tiles of its band from its
// own on. With two workgroups per CU, the busiest slot is taken to share its CU with a
// typical (median) one.
double local_cost(int B, int N, int grid_w, int radius, int ts, int xcds, int slots, int wgs_per_cu, double block_cost)
{
    const int nblk = (N + ts - 1) / ts;
    std::vector<int> tiles(nblk);
    long total = 0;
    for (int t = 0; t < nblk; ++t) {
        const long r_last = (long)(std::min((t + 1) * ts, N) - 1) / grid_w;
        const long thi = std::min<long>(nblk - 1, ((r_last + radius + 1) * (long)grid_w - 1) / ts);
        tiles[t] = (int)(thi - t + 1);
        total += tiles[t];
    }
    const long imgs = (B + xcds - 1) / xcds;  // images of the largest group
    const long items = imgs * nblk;
    if (items > 64L * slots) return (double)imgs * total / slots * wgs_per_cu * block_cost;  // many rounds: balanced
    std::vector<long> load(slots, 0);
    for (long k = 0; k < items; ++k) load[k % slots] += tiles[k % nblk];
    std::sort(load.begin(), load.end());
    const long busiest = load[slots - 1];
    const long typical = load[slots / 2];
    return (double)(wgs_per_cu == 1 ? busiest : busiest + typical) * block_cost;
}

}  // namespace

bool valid_local_block_rows(int requested) { return requested == 0 || requested == kLCT || requested == kPCT; }

int local_block_rows(int B, int N, int D, int dt, int grid_w, int radius, int requested)
{
    if (!use_persistent(D, dt)) return N;
    if (requested != 0) return requested;
    const int cus = device_cus();
    if (cus <= 0) return kPCT;
    const int xcds = (cus % kXcds == 0 && B >= kXcds) ? kXcds : 1;
    const double large = local_cost(B, N, grid_w, radius, kPCT, xcds, cus * kPWGS / xcds, kPWGS, 1.0);
    const double small = local_cost(B, N, grid_w, radius, kLCT, xcds, cus * kLWGS / xcds, kLWGS, kLSmallBlockCost);
    return small < large ? kLCT : kPCT;
}

int partial_tile_width(int B, int D, int dt, int N, int schedule)
{
    if (!use_persistent(D, dt)) return N;
    return small_blocks(B, N, schedule) ? kTCT : kPCT;
}

hipError_t affinity_schedule(int B, int N, int D, int dt, int schedule, int* used)
{
    *used = kScheduleFull;
    if (!use_persistent(D, dt)) return hipSuccess;  // the staged kernel covers every pair
    if (small_blocks(B, N, schedule)) {
        *used = kScheduleFull64;
        return hipSuccess;
    }
    const int cus = device_cus();
    if (cus <= 0) return hipErrorInvalidDevice;
    const int xcds = (cus % kXcds == 0 && B >= kXcds) ? kXcds : 1;
    if (symmetric_schedule(B, N, xcds, cus * kPWGS / xcds, schedule)) *used = kScheduleSymmetric;
    return hipSuccess;
}

hipError_t launch_affinity(const void* x, const int32_t* x_off, int B, int N, int D, int dt, int schedule, float* pv,
                           int32_t* pi, hipStream_t stream, hipEvent_t start, hipEvent_t stop, const float* xinv)
{
    const int T = partial_tiles(N);
    if (xinv && !affinity_takes_norms(D, dt)) return hipErrorInvalidValue;  // those kernels sum their own norms
    if (use_persistent(D, dt)) {
        const int cus = device_cus();
        if (cus <= 0) return hipErrorInvalidDevice;
        // kPWGS workgroups per CU. With a batch of at least 8 images, group the
        // workgroups by XCD.
        const int xcds = (cus % kXcds == 0 && B >= kXcds) ? kXcds : 1;
        const int groups = cus * kPWGS;
        if (small_blocks(B, N, schedule)) {
            if (dt == kBf16)
                launch_persistent<Bf16, kTWC, kTWQ, kTMT, kTNT, false>(x, x_off, xinv, B, N, D, T, xcds, groups, pv, pi,
                                                                        stream, start, stop);
            else
                launch_persistent<F32, kTWC, kTWQ, kTMT, kTNT, false>(x, x_off, xinv, B, N, D, T, xcds, groups, pv, pi,
                                                                       stream, start, stop);
            return hipGetLastError();
        }
        const bool sym = symmetric_schedule(B, N, xcds, groups / xcds, schedule);
        if (dt == kBf16) {
            if (sym)
                launch_persistent<Bf16, kSWC, kSWQ, kSMT, kSNT, true>(x, x_off, xinv, B, N, D, T, xcds, groups, pv, pi,
                                                                       stream, start, stop);
            else
                launch_persistent<Bf16, kPWC, kPWQ, kPMT, kPNT, false>(x, x_off, xinv, B, N, D, T, xcds, groups, pv, pi,
                                                                        stream, start, stop);
        } else {
            if (sym)
                launch_persistent<F32, kSWC, kSWQ, kSMT, kSNT, true>(x, x_off, xinv, B, N, D, T, xcds, groups, pv, pi,
                                                                      stream, start, stop);
            else
                launch_persistent<F32, kPWC, kPWQ, kPMT, kPNT, false>(x, x_off, xinv, B, N, D, T, xcds, groups, pv, pi,
                                                                       stream, start, stop);
        }
        return hipGetLastError();
    }
    if (dt == kBf16) return launch_staged<Bf16, 2, 4, 4, 2, 128>(x, x_off, B, N, D, T, pv, pi, stream, start, stop);
    return launch_staged<F32, 2, 2, 2, 2, 128>(x, x_off, B, N, D, T, pv, pi, stream, start, stop);
}

hipError_t launch_affinity_local(const void* x, const int32_t* x_off, const float* xinv, const int32_t* pos,
                                 int grid_w, int radius, int block_rows,
                                 int B, int N, int D, int dt, float* pv, int32_t* pi, hipStream_t stream,
                                 hipEvent_t start, hipEvent_t stop)
{
    const int T = partial_tiles(N);
    const Window win{pos, grid_w, radius};
    if (use_persistent(D, dt)) {
        // The persistent kernel on the symmetric schedule, one item per query block and the
        // tiles of its band from its own on (given norms: bf16 only), with the block size
        // local_block_rows picks (block_rows: the caller's, 0 to estimate it here).
        const int cus = device_cus();
        if (cus <= 0) return hipErrorInvalidDevice;
        const int xcds = (cus % kXcds == 0 && B >= kXcds) ? kXcds : 1;
        const bool small = local_block_rows(B, N, D, dt, grid_w, radius, block_rows) == kLCT;
        if (small) {
            if (dt == kBf16)
                launch_persistent<Bf16, kLWC, kLWQ, kLMT, kLNT, true, true>(x, x_off, xinv, B, N, D, T, xcds,
                                                                            cus * kLWGS, pv, pi, stream, start, stop,
                                                                            win);
            else
                launch_persistent<F32, kLWC, kLWQ, kLMT, kLNT, true, true>(x, x_off, nullptr, B, N, D, T, xcds,
                                                                           cus * kLWGS, pv, pi, stream, start, stop,
                                                                           win);
        } else if (dt == kBf16) {
            launch_persistent<Bf16, kSWC, kSWQ, kSMT, kSNT, true, true>(x, x_off, xinv, B, N, D, T, xcds, cus * kPWGS,
                                                                        pv, pi, stream, start, stop, win);
        } else {
            launch_persistent<F32, kSWC, kSWQ, kSMT, kSNT, true, true>(x, x_off, nullptr, B, N, D, T, xcds, cus * kPWGS,
                                                                       pv, pi, stream, start, stop, win);
        }
        return hipGetLastError();
    }
    if (dt == kBf16)
        return launch_staged<Bf16, 2, 4, 2, 2, 128, true>(x, x_off, B, N, D, T, pv, pi, stream, start, stop, win);
    return launch_staged<F32, 2, 2, 2, 2, 128, true>(x, x_off, B, N, D, T, pv, pi, stream, start, stop, win);
}

}  // namespace mpm
