// FULL-mode heads (Algorithm 1, first branch): exact softmax attention of a
// head's queries over all N = S * P keys of all views, Y_h =
// softmax(Q_h K_h^T / sqrt(d)) V_h, on MFMA with an online softmax over
// 64-key tiles that are double-buffered through LDS.
//
// Work is taken from the FULL bucket that the mode assignment wrote on the
// device: a grid sized for every head exits early past n_full * q_tiles, so
// no mode is ever copied to the host.
#include <type_traits>

#include "vp_device.hpp"
#include "vp_internal.hpp"

namespace vp {

constexpr int kBK = 64;       // keys per tile

// Number of FULL heads in the bucket array written by the mode assignment,
// 0 if the counts are inconsistent with H (never index past the head list).
__device__ __forceinline__ int full_count(const int32_t* buckets, int H) {
    const int c0 = buckets[0], c1 = buckets[1], c2 = buckets[2];
    if (c0 < 0 || c1 < 0 || c2 < 0 || c0 + c1 + c2 != H) return 0;
    return c2;
}

// Head id of FULL slot `slot` (< full_count), or -1 if out of range.
__device__ __forceinline__ int full_head(const int32_t* buckets, int H, int slot) {
    const int h = buckets[3 + buckets[0] + buckets[1] + slot];
    return (h >= 0 && h < H) ? h : -1;
}
constexpr int kLdsRow = 72;   // bf16 LDS row stride (144 B: 16-B aligned, bank-staggered)

// ------------------------------------------------------------------------
// K5a: the scale of each FULL head's packed values.  The attention
// kernels multiply fp16 weights with fp16 values; the gather stores
// V_h 2^-e_h, with e_h chosen so that the head's largest |v| lies in
// [2^14, 2^15), and the kernels multiply O by 2^e_h at the end (both scalings
// exact).  Every bf16 value then fits fp16's range; values more than 2^29
// below the head's largest land in fp16's subnormals (absolute error at most
// 2^-40 of that largest value).
// K5a: per (group of kVmaxTiles key tiles, FULL slot), max |v|; the gather
// (K5) reduces those per slot and records vsc[slot] = (2^-e_h, 2^e_h).
// ------------------------------------------------------------------------
constexpr int kVmaxTiles = 16;

__device__ __forceinline__ float block_max256(float m, float* red) {
    m = wave_max(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

__global__ __launch_bounds__(256) void k_vmax_partial(const bf16* __restrict__ V,
                                                      const int32_t* __restrict__ buckets,
                                                      int64_t N, int H,
                                                      float* __restrict__ vpart) {
    const int slot = blockIdx.y;
    if (slot >= full_count(buckets, H)) return;
    const int h = full_head(buckets, H, slot);
    if (h < 0) return;
    const int64_t r0 = (int64_t)blockIdx.x * kVmaxTiles * kBK;
    const int64_t r1 = (r0 + kVmaxTiles * kBK < N) ? r0 + kVmaxTiles * kBK : N;
    const int seg = (threadIdx.x & 7) * 8;
    float m = 0.f;
    // Four rows per thread and iteration, their loads issued together.
    for (int64_t row = r0 + (threadIdx.x >> 3); row < r1; row += 128) {
        bf16x8 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t rr = row + 32 * u;
            v[u] = rr < r1 ? load_bf16x8(V + (rr * H + h) * kD + seg) : zero_bf16x8();
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int j = 0; j < 8; ++j) m = fmaxf(m, fabsf(bf16_to_f32(v[u][j])));
    }
    __shared__ float red[4];
    m = block_max256(m, red);
    if (threadIdx.x == 0) vpart[(int64_t)slot * gridDim.x + blockIdx.x] = m;
}

// Exponent e_h of the head's V scale 2^-e_h from its largest |v| (so that
// max |v| 2^-e_h lies in [2^14, 2^15)).  An all-zero head keeps scale 1; an
// infinite value (NaN never wins fmaxf) keeps scale 1 too and reaches the
// output as it would in exact arithmetic.
__device__ __forceinline__ int vscale_exponent(float m) {
    int e = 0;
    if (m > 0.f && m <= 3.4028235e38f) e = ilogbf(m) - 14;
    return e < -126 ? -126 : (e > 126 ? 126 : e);
}

// ------------------------------------------------------------------------
// K5: bucket gather.  For each FULL head (slot s of the FULL bucket), copy
// V_h 2^-e_h into a packed, tile-transposed fp16 buffer Vt[s][tile][d][64
// keys], K_h into packed fp16 tiles Kh[s][tile][64 keys][d] (key rows in
// swap23 order; bf16 values convert exactly while |k| stays in fp16's normal
// range), keys past N zero in both, and record kmax[s][tile] = max |k_j| over
// the tile's keys.  The attention kernels read the tiles as contiguous 8 KB
// blocks whose rows feed the MFMA operands directly, and use kmax to bound
// the logits.
// ------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_gather_vt(const bf16* __restrict__ K,
                                                   const bf16* __restrict__ V,
                                                   const int32_t* __restrict__ buckets, int64_t N,
                                                   int H, int nkt, const float* __restrict__ vpart,
                                                   int nvp, float* __restrict__ vsc,
                                                   f16* __restrict__ Vt, f16* __restrict__ Kh,
                                                   float* __restrict__ kmax) {
    const int slot = blockIdx.y, tile = blockIdx.x;
    const int nfull = full_count(buckets, H);
    if (slot >= nfull) return;
    const int h = full_head(buckets, H, slot);
    if (h < 0) return;
    __shared__ __attribute__((aligned(16))) f16 s[kD * kLdsRow];
    __shared__ float s_norm[4];
    const int t = threadIdx.x;
    const int key = t >> 2, dseg = (t & 3) * 16;
    const int64_t row = (int64_t)tile * kBK + key;
    const bool ok = row < N;
    const int64_t off = ((ok ? row : 0) * H + h) * kD + dseg;
    bf16x8 a = load_bf16x8(V + off), b = load_bf16x8(V + off + 8);
    bf16x8 ka = load_bf16x8(K + off), kb = load_bf16x8(K + off + 8);
    if (!ok) a = b = ka = kb = zero_bf16x8();
    // The head's V scale from the partial maxima (every workgroup of the
    // head reduces the same values in the same order; the tile-0 one
    // records the scale and its inverse for the attention kernels).
    float vm = 0.f;
    for (int i = t; i < nvp; i += 256) vm = fmaxf(vm, vpart[(int64_t)slot * nvp + i]);
    vm = block_max256(vm, s_norm);
    const int e = vscale_exponent(vm);
    const float down = ldexpf(1.f, -e);
    if (tile == 0 && t == 0) {
        vsc[2 * slot] = down;
        vsc[2 * slot + 1] = ldexpf(1.f, e);
    }
    __syncthreads();   // s_norm is reused below
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        s[(dseg + j) * kLdsRow + key] = (f16)(bf16_to_f32(a[j]) * down);
        s[(dseg + 8 + j) * kLdsRow + key] = (f16)(bf16_to_f32(b[j]) * down);
    }
    float n2 = 0.f;
    f16x8 ha, hb;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const float x = bf16_to_f32(ka[j]), y = bf16_to_f32(kb[j]);
        ha[j] = (f16)x;
        hb[j] = (f16)y;
        n2 = fmaf(x, x, fmaf(y, y, n2));
    }
    f16* kd = Kh + (((int64_t)slot * nkt + tile) * kBK + swap23(key)) * kD + dseg;
    *reinterpret_cast<f16x8*>(kd) = ha;
    *reinterpret_cast<f16x8*>(kd + 8) = hb;
    n2 += __shfl_xor(n2, 1);
    n2 += __shfl_xor(n2, 2);
    n2 = wave_max(n2);
    if ((t & 63) == 0) s_norm[t >> 6] = n2;
    __syncthreads();
    if (t == 0)
        kmax[(int64_t)slot * nkt + tile] =
            sqrtf(fmaxf(fmaxf(s_norm[0], s_norm[1]), fmaxf(s_norm[2], s_norm[3])));
    const int d = t >> 2, kseg = (t & 3) * 16;
    f16* dst = Vt + (((int64_t)slot * nkt + tile) * kD + d) * kBK + kseg;
    *reinterpret_cast<f16x8*>(dst) = *reinterpret_cast<const f16x8*>(&s[d * kLdsRow + kseg]);
    *reinterpret_cast<f16x8*>(dst + 8) =
        *reinterpret_cast<const f16x8*>(&s[d * kLdsRow + kseg + 8]);
}

// ------------------------------------------------------------------------
// K6 (bf16): FULL-head attention.  Per 64-key tile and wave of 64 queries:
// S^T = K Q^T (keys x queries, 2 x 2 blocks of 32x32, 16 MFMAs), softmax
// weights in registers, O^T += V^T P^T (d x queries, 16 MFMAs).  Each lane
// owns one query column of every block, so softmax row statistics stay in
// the lane plus one exchange with lane ^ 32.  K rows sit in LDS with index
// bits 2 and 3 swapped so that the S^T registers hold eight consecutive keys
// per lane-half: they become the B operand of the PV MFMA without any data
// movement.  Operands are fp16: K as packed by the gather (bf16 values in
// fp16's range convert exactly), V^T scaled by 2^-e_h, P rounded to nearest
// (relative error at most 2^-11).
//
// Softmax is invariant to the reference point subtracted from the logits
// before exponentiation.  A work item (512 queries of one head) runs in one
// of three modes, chosen from Cauchy-Schwarz bounds (|q . k| <= |q| max_j
// |k_j|) before its first tile:
//  - FAST: every logit of the item lies within +-kFastBound in log2 units.
//    The scale c = log2(e) / sqrt(d) is folded into Q (rounded to fp16,
//    relative error 2^-11), S comes out of the MFMA in log2 units and the
//    reference point is 0: p = 2^S lies in [2^-10, 2^10], fp16's normal range,
//    and a score costs one exp2 and half a pack.
//  - EXT: every logit lies within +-kExtBound.  Q and S as in FAST mode, and
//    the reference point m of a query stays 0 unless the segment's first
//    tile's maximum lies below kExtLow (then m is that maximum) or a weight
//    or a lane's fp16 row sum overflows (then m moves to the tile maximum,
//    O and l are rescaled and the tile's weights taken again).  While m = 0
//    for every query of a wave's 32-query block, its scores cost what they
//    cost in FAST mode; otherwise one subtraction more.  The fp16 rounding
//    of c q moves a logit by at most 2^-11 kExtBound.
//  - WIDE: Q keeps its bf16 value (exact in fp16), logits are scaled in fp32
//    and a running reference point m moves with the logits.  The segment's
//    first tile sets m to its maximum; every later tile is exponentiated
//    against m as it comes, and only if a weight or a lane's fp16 row sum
//    overflows (some logit more than ~15 above m) is the tile maximum taken,
//    m moved to it (O and l rescaled) and the tile's weights taken again.
//    A score costs one FMA more than in FAST mode.  (Teacher instances keep
//    the earlier test before the weights: a tile whose logits provably stay
//    below m + kSlack, by its largest key norm, is exponentiated against m
//    directly; otherwise the tile maximum is taken and m moves when the tile
//    exceeds m + kSlack.)
// In EXT and WIDE modes one wave-wide vote per tile, after both of a wave's
// 32-query blocks are packed and summed, decides whether any of them
// overflowed.
// Row sums: the packed fp16 weights of a lane's 32 keys per tile are added
// as a tree of packed fp16 adds (at most 32 weights of at most 2^10: no
// overflow; relative error at most 5 * 2^-11), then into l in fp32.  The
// numerator uses the same rounded weights.  Teacher instances (which also
// write each query's log2 sum_k 2^x) run every item in WIDE mode, whose
// logits are exact, and add the unrounded fp32 weights with a compensated
// sum instead.  Items whose Q or K values exceed fp16's range are flagged
// and left to K6b, which keeps bf16 operands.
// ------------------------------------------------------------------------
constexpr int kBQ16 = 256;
constexpr float kFastBound = 10.f;   // |logit| bound (log2 units) of FAST mode
constexpr float kSlack = 10.f;       // WIDE: log2 headroom above the running reference
constexpr float kF16Safe = 4096.f;   // FAST: |c q|, |k| limit for the fp16 operands
constexpr float kF16Max = 65504.f;   // WIDE: largest finite fp16
constexpr float kExtBound = 24.f;    // EXT: |logit| bound (log2 units)
constexpr float kExtLow = -4.f;      // EXT: lowest first-tile maximum kept at reference 0

// Kahan step: adds x to the sum s with compensation e (the sum is s - e).
__device__ __forceinline__ void kahan_add(float& s, float& e, float x) {
    const float y = x - e;
    const float t = s + y;
    e = (t - s) - y;
    s = t;
}

__device__ __forceinline__ float dot2_ones(uint32_t pair, float acc) {
    const f16x2 v = __builtin_bit_cast(f16x2, pair);
    const f16x2 one = {(f16)1.0f, (f16)1.0f};
    return __builtin_amdgcn_fdot2(v, one, acc, false);
}

// Sum of the 32 packed fp16 weights of one query block (16 registers of two
// weights) as a tree of packed fp16 adds, added to acc in fp32.
__device__ __forceinline__ float tree_sum(const f16x8 (&P)[2][2], float acc) {
    f16x2 t[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        t[2 * i] = f16x2{P[0][0][2 * i], P[0][0][2 * i + 1]} +
                   f16x2{P[0][1][2 * i], P[0][1][2 * i + 1]};
        t[2 * i + 1] = f16x2{P[1][0][2 * i], P[1][0][2 * i + 1]} +
                       f16x2{P[1][1][2 * i], P[1][1][2 * i + 1]};
    }
#pragma unroll
    for (int w = 4; w >= 1; w >>= 1)
#pragma unroll
        for (int i = 0; i < w; ++i) t[i] = t[i] + t[i + w];
    return dot2_ones(__builtin_bit_cast(uint32_t, t[0]), acc);
}

// Y[q, h, d] = O up / l for the wave's two 32-query blocks (up = 2^e_h, the
// inverse of the packed values' scale); lane holds d = 32 db + 8 g + 4 hh + i
// for i = 0..3.
__device__ __forceinline__ void store_rows(const f32x16 (&O)[2][2], const float (&l)[2],
                                           const int64_t (&qidx)[2], int64_t N, int H, int h,
                                           int hh, float up, void* __restrict__ Y, int ydt) {
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const float lt = l[qb] + __shfl_xor(l[qb], 32);
        const float inv = up / lt;
        const int64_t qi = qidx[qb];
        if (qi < N) {
#pragma unroll
            for (int db = 0; db < 2; ++db)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int64_t off = (qi * H + h) * kD + db * 32 + 8 * g + 4 * hh;
                    const float y0 = O[qb][db][4 * g] * inv, y1 = O[qb][db][4 * g + 1] * inv;
                    const float y2 = O[qb][db][4 * g + 2] * inv, y3 = O[qb][db][4 * g + 3] * inv;
                    if (ydt == DT_BF16) {
                        bf16x4 v;
                        v[0] = (bf16)y0; v[1] = (bf16)y1; v[2] = (bf16)y2; v[3] = (bf16)y3;
                        *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(Y) + off) = v;
                    } else {
                        *reinterpret_cast<float4*>(reinterpret_cast<float*>(Y) + off) =
                            make_float4(y0, y1, y2, y3);
                    }
                }
        }
    }
}

// o_q = m + log2 l per query of the wave's two blocks (teacher instances).
// (m is the same in both lane halves.)
__device__ __forceinline__ void store_offsets(const float (&l)[2], const float (&m)[2],
                                              const int64_t (&qidx)[2], int64_t N, int h, int hh,
                                              float* __restrict__ off) {
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const float lt = l[qb] + __shfl_xor(l[qb], 32);
        if (hh == 0 && qidx[qb] < N) off[(int64_t)h * N + qidx[qb]] = m[qb] + __log2f(lt);
    }
}

// K6a: one workgroup = 8 waves x 64 queries of one FULL head, two waves per
// SIMD (waves w and w + 4).  Ping-pong: waves 0-3 (group A) and 4-7 (group
// B) run the same sequence of phases, matrix(0), vector(0), matrix(1), ...,
// group B one phase behind, with one workgroup barrier per phase, so that in
// every phase one wave of each SIMD issues MFMAs while the other issues the
// softmax's vector instructions:
//   matrix(t): O += V(t-1) P(t-1)  then  S(t) = K(t) Q^T   (32 MFMAs)
//   vector(t): P(t) = fp16 weights of S(t), l += their row sums
// LDS slot t % 2 holds K(t) and V(t-1).
//
// Balanced tail: the work is n_full x q-tiles items of nkt key tiles.  A
// fixed grid of G workgroups (one per CU) takes the items in rounds,
// workgroup w item r G + w, so that in every round the workgroups of an XCD
// stream the same key tiles of one head through its L2.  The R < G items of
// the last, partial round are cut into one flat sequence of R nkt item-tile
// steps, split evenly over the workgroups (at least kMinPartTiles steps
// each), so the tail takes R / G of a round instead of a whole one.  Results
// over key ranges combine exactly: a workgroup that covers only part of an
// item writes its unnormalized O, l and reference point m to one of its two
// partial slots (0 for the first item of its range, 1 for the last), and K6c
// combines the parts of each split item in workgroup order.  The part
// holding tile 0 writes exact_items[L] (1 = left to K6b), so flags never
// carry over.
constexpr int kBQf = 512;
constexpr int kStreamWG = 256;      // grid: one workgroup per CU
constexpr int kPartFloats = kBQf * kD + 2 * kBQf;   // partial slot: O[512][64], l[512], m[512]

constexpr int kMinPartTiles = 8;    // fewest key tiles per workgroup in the tail
constexpr int64_t kRotateTiles = 4096;   // 64 MB of K and V^T tiles (16 KB each)

// Workgroups used for T tail steps (at most G, at least kMinPartTiles steps
// each), the first step of workgroup w, and the workgroup holding step x.
__device__ __forceinline__ int tail_groups(int64_t T, int G) {
    const int64_t g = T / kMinPartTiles;
    return g < 1 ? 1 : (g < G ? (int)g : G);
}
__device__ __forceinline__ int64_t tail_start(int w, int64_t T, int G) {
    return (int64_t)w * T / G;
}
__device__ __forceinline__ int tail_owner(int64_t x, int64_t T, int G) {
    return (int)(((x + 1) * G + T - 1) / T) - 1;
}

enum { ITEM_FAST = 0, ITEM_WIDE = 1, ITEM_EXACT = 2, ITEM_EXT = 3 };

template <bool kTeach>
__global__ __launch_bounds__(512, 1) void k_flash_bf16(const bf16* __restrict__ Q,
                                                       const f16* __restrict__ Kh,
                                                       const f16* __restrict__ Vt,
                                                       const float* __restrict__ kmax,
                                                       const float* __restrict__ vsc,
                                                       const int32_t* __restrict__ buckets,
                                                       int64_t N, int H, int nqt, int nkt, float c,
                                                       int32_t* __restrict__ exact_items,
                                                       float* __restrict__ part, int G,
                                                       void* __restrict__ Y, int ydt,
                                                       float* __restrict__ off) {
    const int nfull = full_count(buckets, H);
    const int active = nfull * nqt;
    if (active == 0) return;
    const int w = xcd_remap(blockIdx.x, G);
    const int full = active / G * G, R = active - full;
    // The wave index is uniform within a wave: say so, so that the group
    // choice and everything derived from it stay scalar.
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int n = lane & 31, hh = lane >> 5;
    const bool groupB = wave >= 4;

    __shared__ __attribute__((aligned(16))) f16 sK[2][kBK * kLdsRow];
    __shared__ __attribute__((aligned(16))) f16 sV[2][kD * kLdsRow];
    __shared__ float sKmax[8], sQmax[8];

    // One segment: key tiles [t0, t1) of item L; written to partial slot
    // pslot of this workgroup if the segment is not the whole item.
    auto segment = [&](int L, int t0, int t1, int pslot) __attribute__((always_inline)) {
        const int slot = L / nqt, qt = L - slot * nqt;
        const int h = full_head(buckets, H, slot);
        if (h < 0) return;

        // max_j |k_j| over the head, from the per-tile maxima.
        const float* kmx = kmax + (int64_t)slot * nkt;
        {
            float km = 0.f;
            for (int i = threadIdx.x; i < nkt; i += 512) km = fmaxf(km, kmx[i]);
            km = wave_max(km);
            if (lane == 0) sKmax[wave] = km;
        }

        // This wave's two 32-query blocks (bf16) and |q| per query.
        bf16x8 qraw[2][4];
        int64_t qidx[2];
        float qn[2];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            const int64_t qi = (int64_t)qt * kBQf + wave * 64 + qb * 32 + n;
            qidx[qb] = qi;
            const bool ok = qi < N;
            const bf16* qp = Q + ((ok ? qi : 0) * H + h) * kD + 8 * hh;
            float n2 = 0.f;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                qraw[qb][ks] = ok ? load_bf16x8(qp + 16 * ks) : zero_bf16x8();
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const float x = bf16_to_f32(qraw[qb][ks][j]);
                    n2 = fmaf(x, x, n2);
                }
            }
            n2 += __shfl_xor(n2, 32);
            qn[qb] = sqrtf(n2);
        }
        {
            const float qm = wave_max(fmaxf(qn[0], qn[1]));
            if (lane == 0) sQmax[wave] = qm;
        }
        __syncthreads();
        int mode;
        {
            float km = sKmax[0], qm = sQmax[0];
#pragma unroll
            for (int v = 1; v < 8; ++v) {
                km = fmaxf(km, sKmax[v]);
                qm = fmaxf(qm, sQmax[v]);
            }
            // Conditions written as "within" so that a NaN norm goes to K6b.
            const bool safe = !kTeach && qm * c <= kF16Safe && km <= kF16Safe;
            const bool fast = safe && qm * c * km <= kFastBound;
            const bool ext = safe && qm * c * km <= kExtBound;
            const bool wide = qm <= kF16Max && km <= kF16Max;
            mode = fast ? ITEM_FAST : (ext ? ITEM_EXT : (wide ? ITEM_WIDE : ITEM_EXACT));
        }
        if (t0 == 0 && threadIdx.x == 0) exact_items[L] = mode == ITEM_EXACT;
        if (mode == ITEM_EXACT) return;   // uniform over the workgroup

        // Q^T operands, kept in registers: fp16 c q (FAST, EXT) or fp16 q
        // (WIDE).
        f16x8 Qop[2][4];
        const float qs = mode == ITEM_WIDE ? 1.f : c;
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    Qop[qb][ks][j] = (f16)(bf16_to_f32(qraw[qb][ks][j]) * qs);

        // Tile copies: group A (threads 0-255) copies K tiles, group B V^T
        // tiles, each a contiguous 8 KB block: 64 rows x 4 segments of 16
        // elements.  r counts tiles from t0.
        const int ns = t1 - t0;
        const int tl = threadIdx.x & 255, lr = tl >> 2, lc = (tl & 3) * 16;
        const f16* Khh = Kh + ((int64_t)slot * nkt + t0) * kBK * kD;
        const f16* Vth = Vt + ((int64_t)slot * nkt + t0) * kD * kBK;
        u32x4 g0, g1;
        // While all FULL heads' tiles fit in 64 MB (a quarter of the
        // last-level cache), the segment's tiles are taken in a rotated
        // order, starting at a different tile in each of the 32 workgroups of
        // an XCD, so that they do not all read the same tile at the same time
        // (larger sets are read in step, so that the workgroups of an XCD
        // share what its L2 holds).
        const int rot = (int64_t)nfull * nkt <= kRotateTiles
                            ? (int)(((int64_t)(w & 31) * ns) >> 5) : 0;
        auto tile_of = [&](int r) {   // r < ns
            const int t = r + rot;
            return t >= ns ? t - ns : t;
        };
        auto fetch = [&](int r) {   // tile r (clamped to the last one) into registers
            r = tile_of(r < ns ? r : ns - 1);
            const u32x4* src = groupB
                ? reinterpret_cast<const u32x4*>(Vth + ((int64_t)r * kD + lr) * kBK + lc)
                : reinterpret_cast<const u32x4*>(Khh + ((int64_t)r * kBK + lr) * kD + lc);
            g0 = src[0];
            g1 = src[1];
        };
        auto stash = [&](int sl) {   // ... into LDS slot sl
            u32x4* dst = groupB ? reinterpret_cast<u32x4*>(&sV[sl][lr * kLdsRow + lc])
                                : reinterpret_cast<u32x4*>(&sK[sl][lr * kLdsRow + lc]);
            dst[0] = g0;
            dst[1] = g1;
        };

        f32x16 O[2][2], S[2][2];
        f16x8 P[2][2][2];
        float l[2], le[2], m[2];   // le: Kahan compensation of l (teacher instances)
        const float qnc[2] = {qn[0] * c, qn[1] * c};
        const f16x8 zp = {};
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            O[qb][0] = O[qb][1] = zero_f32x16();
            l[qb] = le[qb] = 0.f;
            m[qb] = mode == ITEM_WIDE ? -INFINITY : 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) P[qb][kb][0] = P[qb][kb][1] = zp;
        }

        // Matrix phase of tile r: O += V(r-1) P(r-1), then S(r) = K(r) Q^T
        // from sK[r%2].  The V operands were read into registers at the end of
        // the wave's previous vector phase, so the 16 PV MFMAs start at once
        // and hide the latency of the K reads.  (PV first: P(r-1) is dead
        // before S(r) is written, so the two can share registers.  r = 0: P
        // and the V operands are zero, so the PV adds exactly nothing.)
        f16x8 va[2][2][2];
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) va[db][kb][0] = va[db][kb][1] = zp;
        auto prefetch_v = [&](int sl) {   // V operands of the next PV product
#pragma unroll
            for (int db = 0; db < 2; ++db)
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int b = 0; b < 2; ++b)
                        va[db][kb][b] = *reinterpret_cast<const f16x8*>(
                            &sV[sl][(db * 32 + n) * kLdsRow + kb * 32 + 16 * b + 8 * hh]);
        };
        auto pv = [&] {
#pragma unroll
            for (int db = 0; db < 2; ++db)
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int b = 0; b < 2; ++b) {
                        O[0][db] = mfma_f16(va[db][kb][b], P[0][kb][b], O[0][db]);
                        O[1][db] = mfma_f16(va[db][kb][b], P[1][kb][b], O[1][db]);
                    }
        };
        auto mma_phase = [&](int r) {
            const int sl = r & 1;
            f16x8 ka[2][4];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int ks = 0; ks < 4; ++ks)
                    ka[kb][ks] = *reinterpret_cast<const f16x8*>(
                        &sK[sl][(kb * 32 + n) * kLdsRow + 16 * ks + 8 * hh]);
            pv();
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    if (ks == 0) S[0][kb] = S[1][kb] = zero_f32x16();
                    S[0][kb] = mfma_f16(ka[kb][ks], Qop[0][ks], S[0][kb]);
                    S[1][kb] = mfma_f16(ka[kb][ks], Qop[1][ks], S[1][kb]);
                }
            // K operands first, then the PV and S products.
            __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 32, 0);
        };
        // Vector phase of tile r: S(r) -> P(r), l += row sums.  The segment's
        // last tile masks keys >= N to weight 0 (a separate instance, so that
        // no other tile pays for the test).
        auto tile_max = [&](int qb) {   // largest S of the tile, per query
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) mx = fmaxf(mx, S[qb][kb][i]);
            return fmaxf(mx, __shfl_xor(mx, 32));
        };
        auto valu_phase = [&](int r, auto last_tag, auto mode_tag, auto mid) {
            constexpr bool kWide = decltype(mode_tag)::value == ITEM_WIDE;
            constexpr bool kExt = decltype(mode_tag)::value == ITEM_EXT;
            (void)last_tag;
            const int tr = t0 + tile_of(r);
            if ((N & (kBK - 1)) && tr == nkt - 1) {
                const int64_t k0 = (int64_t)tr * kBK;
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int64_t key = k0 + kb * 32 + 16 * (i >> 3) + 8 * hh + (i & 7);
                        if (key >= N) S[0][kb][i] = S[1][kb][i] = -INFINITY;
                    }
            }
            const float kbt = kTeach ? kmx[tr] : 0.f;
            if (kExt) {
                // Exponentials in place (S <= kExtBound - m: finite in fp32),
                // then fp16 packs and row sums; a query block whose weights
                // or row sums overflow fp16 moves its reference point to the
                // tile maximum, log2 of its largest exponential.
                bool sh[2];
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) {
                    if (r == 0) {
                        const float mx = tile_max(qb);
                        m[qb] = mx < kExtLow ? mx : 0.f;   // O, l are still 0
                    }
                    sh[qb] = __builtin_amdgcn_ballot_w64(m[qb] != 0.f) != 0;
                }
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) {
                    const float nm = -m[qb];
                    if (sh[qb]) {
#pragma unroll
                        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                            for (int i = 0; i < 16; ++i)
                                S[qb][kb][i] = exp2f_fast(S[qb][kb][i] + nm);
                    } else {
#pragma unroll
                        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                            for (int i = 0; i < 16; ++i) S[qb][kb][i] = exp2f_fast(S[qb][kb][i]);
                    }
                }
                auto pack = [&](int qb, float sc) {   // P = fp16 (sc * e)
#pragma unroll
                    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                        for (int b = 0; b < 2; ++b) {
                            u32x4 pk;
#pragma unroll
                            for (int j = 0; j < 4; ++j) {
                                f32x2 e = {S[qb][kb][8 * b + 2 * j], S[qb][kb][8 * b + 2 * j + 1]};
                                if (sc != 1.f) e = e * sc;
                                pk[j] = __builtin_bit_cast(uint32_t,
                                                           __builtin_convertvector(e, f16x2));
                            }
                            P[qb][kb][b] = __builtin_bit_cast(f16x8, pk);
                        }
                };
                // Both blocks packed and summed, then one overflow test for
                // the two (a branch per block would keep the second block's
                // work from overlapping the first one's dependent sums).
                float ln[2];
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) pack(qb, 1.f);
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) ln[qb] = tree_sum(P[qb], l[qb]);
                if (__builtin_amdgcn_ballot_w64(!(ln[0] < INFINITY) || !(ln[1] < INFINITY)) != 0) {
#pragma unroll
                    for (int qb = 0; qb < 2; ++qb) {
                        if (__builtin_amdgcn_ballot_w64(!(ln[qb] < INFINITY)) != 0) {
                            const float mn = fmaxf(m[qb], m[qb] + __log2f(tile_max(qb)));
                            const float al = exp2f_fast(m[qb] - mn);
                            m[qb] = mn;
                            l[qb] *= al;
#pragma unroll
                            for (int db = 0; db < 2; ++db)
#pragma unroll
                                for (int i = 0; i < 16; ++i) O[qb][db][i] *= al;
                            pack(qb, al);
                            ln[qb] = tree_sum(P[qb], l[qb]);
                        }
                    }
                }
                l[0] = ln[0];
                l[1] = ln[1];
                // (S is dead: the next V operands' LDS reads)
                mid();
                return;
            }
            if (!kWide && !kTeach) {
                // FAST: all exponentials first (in place), then the packs and
                // row sums.
#pragma unroll
                for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                        for (int i = 0; i < 16; ++i) S[qb][kb][i] = exp2f_fast(S[qb][kb][i]);
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) {
#pragma unroll
                    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                        for (int b = 0; b < 2; ++b) {
                            u32x4 pk;
#pragma unroll
                            for (int j = 0; j < 4; ++j) {
                                const f32x2 e = {S[qb][kb][8 * b + 2 * j],
                                                 S[qb][kb][8 * b + 2 * j + 1]};
                                pk[j] = __builtin_bit_cast(uint32_t,
                                                           __builtin_convertvector(e, f16x2));
                            }
                            P[qb][kb][b] = __builtin_bit_cast(f16x8, pk);
                        }
                }
                // (S is dead: the next V operands' LDS reads go here, so that
                // they complete under the row sums rather than at the barrier.)
                mid();
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) l[qb] = tree_sum(P[qb], l[qb]);
                return;
            }
            // WIDE items and teacher instances from here on.  WIDE (not
            // teacher): the segment's first tile sets m to its maximum before
            // the weights; later tiles are taken against m and redone only on
            // fp16 overflow (below).
            auto reset_m = [&](int qb) {
                float mx = -INFINITY;
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int i = 0; i < 16; ++i) mx = fmaxf(mx, S[qb][kb][i]);
                mx = fmaxf(mx, __shfl_xor(mx, 32)) * c;
                const float mn = fmaxf(m[qb], mx);
                const float al = exp2f_fast(m[qb] - mn);
                m[qb] = mn;
                l[qb] *= al;
#pragma unroll
                for (int db = 0; db < 2; ++db)
#pragma unroll
                    for (int i = 0; i < 16; ++i) O[qb][db][i] *= al;
            };
            if (!kTeach && r == 0) {
                reset_m(0);
                reset_m(1);
            }
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                if (kTeach) {
                    // Keep m unless the bound cannot rule out a logit above
                    // m + kSlack for some query of this block.
                    if (__builtin_amdgcn_ballot_w64(qnc[qb] * kbt > m[qb] + kSlack) != 0) {
                        float mx = -INFINITY;
#pragma unroll
                        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                            for (int i = 0; i < 16; ++i) mx = fmaxf(mx, S[qb][kb][i]);
                        mx = fmaxf(mx, __shfl_xor(mx, 32)) * c;
                        const bool move = mx > m[qb] + kSlack;
                        const float mn = move ? mx : m[qb];
                        const float al = move ? exp2f_fast(m[qb] - mn) : 1.f;
                        m[qb] = mn;
                        l[qb] *= al;
                        le[qb] *= al;
#pragma unroll
                        for (int db = 0; db < 2; ++db)
#pragma unroll
                            for (int i = 0; i < 16; ++i) O[qb][db][i] *= al;
                    }
                }
                const float nm = -m[qb];
                float ls0 = 0.f, ls1 = 0.f;
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int b = 0; b < 2; ++b) {
                        u32x4 pk;
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            f32x2 e;
                            e[0] = exp2f_fast(fmaf(S[qb][kb][8 * b + 2 * j], c, nm));
                            e[1] = exp2f_fast(fmaf(S[qb][kb][8 * b + 2 * j + 1], c, nm));
                            pk[j] = __builtin_bit_cast(uint32_t,
                                                       __builtin_convertvector(e, f16x2));
                            if (kTeach) {
                                ls0 += e[0];
                                ls1 += e[1];
                            }
                        }
                        P[qb][kb][b] = __builtin_bit_cast(f16x8, pk);
                    }
                if (kTeach) {
                    kahan_add(l[qb], le[qb], ls0 + ls1);
                    if (qb == 0) mid();   // (the first block's S is dead)
                }
            }
            if (kTeach) return;
            // WIDE: both blocks' fp16 row sums, then one overflow vote for
            // the two (as in EXT mode); a block that overflowed moves m to
            // its tile maximum and is taken again from its fp32 logits.
            float ln[2];
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) ln[qb] = tree_sum(P[qb], l[qb]);
            if (__builtin_amdgcn_ballot_w64(!(ln[0] < INFINITY) || !(ln[1] < INFINITY)) != 0) {
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) {
                    if (__builtin_amdgcn_ballot_w64(!(ln[qb] < INFINITY)) == 0) continue;
                    reset_m(qb);
                    const float nm2 = -m[qb];
#pragma unroll
                    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                        for (int b = 0; b < 2; ++b) {
                            u32x4 pk;
#pragma unroll
                            for (int j = 0; j < 4; ++j) {
                                f32x2 e;
                                e[0] = exp2f_fast(fmaf(S[qb][kb][8 * b + 2 * j], c, nm2));
                                e[1] = exp2f_fast(fmaf(S[qb][kb][8 * b + 2 * j + 1], c, nm2));
                                pk[j] = __builtin_bit_cast(uint32_t,
                                                           __builtin_convertvector(e, f16x2));
                            }
                            P[qb][kb][b] = __builtin_bit_cast(f16x8, pk);
                        }
                    ln[qb] = tree_sum(P[qb], l[qb]);
                }
            }
            l[0] = ln[0];
            l[1] = ln[1];
            mid();   // (S is dead)
        };
        const std::false_type body{};
        const std::true_type tail{};
        // End of a phase: a workgroup barrier that the compiler may not
        // schedule any instruction across (it would otherwise hoist the next
        // phase's register-only work above it and undo the alternation).
        auto phase_end = [] {
            __builtin_amdgcn_sched_barrier(0);
            __syncthreads();
            __builtin_amdgcn_sched_barrier(0);
        };

        // Phases, one workgroup barrier each (2 ns + 2 in both groups, counting
        // the prologue's):
        //   group A:  M(0) V(0) M(1) V(1) ... M(ns-1) V(ns-1) -
        //   group B:  -    M(0) V(0) M(1) ... V(ns-2) M(ns-1) V(ns-1)
        // A wave issues its 32 MFMAs in a few dozen cycles and then waits for
        // the other wave's vector phase, so the tile copies live in the
        // matrix phases: a group loads a tile from global memory during its
        // vector phase and stores it to LDS after issuing the MFMAs of its
        // next matrix phase.  Group A stores K(r+1) to sK[(r+1) % 2] during
        // M(r); group B stores V(r+1) to sV[r % 2] during M(r) (V(0) to sV[1]
        // in the first phase), two phases before group A reads those V
        // operands at the end of its V(r+1) for M(r+2), and group B at the end
        // of its own V(r+1).  A slot is rewritten only after both groups'
        // last reads.
        auto mma_then = [&](int r, int store_slot) {
            mma_phase(r);
            __builtin_amdgcn_sched_barrier(0);
            if (store_slot >= 0) stash(store_slot);
        };
        auto run = [&](auto mode_tag) {
            if (!groupB) {
                fetch(0);
                stash(0);
                fetch(1);
                phase_end();
                for (int r = 0; r < ns - 1; ++r) {
                    mma_then(r, (r + 1) & 1);
                    phase_end();
                    fetch(r + 2);
                    valu_phase(r, body, mode_tag, [&] { prefetch_v((r + 1) & 1); });
                    phase_end();
                }
                mma_then(ns - 1, -1);
                phase_end();
                valu_phase(ns - 1, tail, mode_tag, [&] { prefetch_v(ns & 1); });
                phase_end();
                phase_end();
            } else {
                fetch(0);
                phase_end();
                stash(1);
                fetch(1);
                phase_end();
                for (int r = 0; r < ns - 1; ++r) {
                    mma_then(r, r & 1);
                    phase_end();
                    fetch(r + 2);
                    valu_phase(r, body, mode_tag, [&] { prefetch_v((r + 1) & 1); });
                    phase_end();
                }
                mma_then(ns - 1, -1);
                phase_end();
                valu_phase(ns - 1, tail, mode_tag, [&] { prefetch_v(ns & 1); });
                phase_end();
            }
            pv();   // O += V(ns-1) P(ns-1)
        };
        if (kTeach || mode == ITEM_WIDE)
            run(std::integral_constant<int, ITEM_WIDE>{});
        else if (!kTeach && mode == ITEM_EXT)
            run(std::integral_constant<int, ITEM_EXT>{});
        else
            run(std::integral_constant<int, ITEM_FAST>{});

        if (kTeach) {
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) l[qb] -= le[qb];
        }
        if (t0 == 0 && t1 == nkt) {
            store_rows(O, l, qidx, N, H, h, hh, vsc[2 * slot + 1], Y, ydt);
            if (kTeach) store_offsets(l, m, qidx, N, h, hh, off);
        } else {
            // Partial slot: O[q][d] unnormalized, then l[q], then m[q]
            // (q = row in item).
            float* ps = part + (int64_t)(w * 2 + pslot) * kPartFloats;
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                const int qr = wave * 64 + qb * 32 + n;
#pragma unroll
                for (int db = 0; db < 2; ++db)
#pragma unroll
                    for (int g = 0; g < 4; ++g)
                        *reinterpret_cast<float4*>(ps + qr * kD + db * 32 + 8 * g + 4 * hh) =
                            make_float4(O[qb][db][4 * g], O[qb][db][4 * g + 1],
                                        O[qb][db][4 * g + 2], O[qb][db][4 * g + 3]);
                const float lt = l[qb] + __shfl_xor(l[qb], 32);
                if (hh == 0) {
                    ps[kBQf * kD + qr] = lt;
                    ps[kBQf * kD + kBQf + qr] = m[qb];
                }
            }
        }
    };

    for (int L = w; L < full; L += G) {
        segment(L, 0, nkt, 0);
        __syncthreads();   // LDS is reused by the next segment
    }
    if (R > 0) {
        const int64_t T = (int64_t)R * nkt;
        const int Gt = tail_groups(T, G);
        if (w < Gt) {
            const int64_t start = tail_start(w, T, Gt), end = tail_start(w + 1, T, Gt);
            for (int64_t x = start; x < end;) {
                const int i = (int)(x / nkt);
                const int t0 = (int)(x - (int64_t)i * nkt);
                const int64_t left = end - x;
                const int t1 = (int64_t)(nkt - t0) < left ? nkt : (int)(t0 + left);
                segment(full + i, t0, t1, x == start ? 0 : 1);
                x += t1 - t0;
                __syncthreads();
            }
        }
    }
}

// K6c: Y of the tail items that K6a split over workgroups: the parts' O and
// l, each relative to its part's reference point m, scaled to the largest m
// and added in workgroup order (fixed, so results are deterministic), then
// O 2^e_h / l.  One workgroup of 256 threads per (tail item, 64-query
// block): 4 threads per query, 16 consecutive values each, so a query's
// 256-byte row of a part is read whole.  Items that K6a finished whole or
// left to K6b exit at once.
constexpr int kCombRows = 64;
__global__ __launch_bounds__(256) void k_flash_combine(const int32_t* __restrict__ buckets,
                                                       int64_t N, int H, int nqt, int nkt,
                                                       const int32_t* __restrict__ exact_items,
                                                       const float* __restrict__ part,
                                                       const float* __restrict__ vsc, int G,
                                                       void* __restrict__ Y, int ydt,
                                                       float* __restrict__ off) {
    const int nfull = full_count(buckets, H);
    const int active = nfull * nqt;
    const int full = active / G * G, R = active - full;
    const int i = blockIdx.x / (kBQf / kCombRows), rb = blockIdx.x % (kBQf / kCombRows);
    if (i >= R) return;
    const int64_t T = (int64_t)R * nkt;
    const int Gt = tail_groups(T, G);
    const int wf = tail_owner((int64_t)i * nkt, T, Gt);
    const int wl = tail_owner((int64_t)(i + 1) * nkt - 1, T, Gt);
    const int L = full + i;
    if (wf == wl || exact_items[L]) return;
    const int slot = L / nqt, qt = L - slot * nqt;
    const int h = full_head(buckets, H, slot);
    if (h < 0) return;
    // partial slot of workgroup v for this item
    auto pslot = [&](int v) {
        const int k = i == (int)(tail_start(v, T, Gt) / nkt) ? 0 : 1;
        return part + (int64_t)(v * 2 + k) * kPartFloats;
    };
    const int qr = rb * kCombRows + (threadIdx.x >> 2), d0 = (threadIdx.x & 3) * 16;
    const int64_t qi = (int64_t)qt * kBQf + qr;
    if (qi >= N) return;
    float mt = -INFINITY;
    for (int v = wf; v <= wl; ++v) mt = fmaxf(mt, pslot(v)[kBQf * kD + kBQf + qr]);
    float lt = 0.f;
    float acc[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) acc[k] = 0.f;
    for (int v = wf; v <= wl; ++v) {
        const float* ps = pslot(v);
        // 2^(m_v - max m): exactly 1 for parts at the largest reference point
        // (every part of a FAST item has m = 0).
        const float sc = exp2f_fast(ps[kBQf * kD + kBQf + qr] - mt);
        lt = fmaf(ps[kBQf * kD + qr], sc, lt);
        const float4* src = reinterpret_cast<const float4*>(ps + qr * kD + d0);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float4 a = src[k];
            acc[4 * k] = fmaf(a.x, sc, acc[4 * k]);
            acc[4 * k + 1] = fmaf(a.y, sc, acc[4 * k + 1]);
            acc[4 * k + 2] = fmaf(a.z, sc, acc[4 * k + 2]);
            acc[4 * k + 3] = fmaf(a.w, sc, acc[4 * k + 3]);
        }
    }
    if (off && d0 == 0) off[(int64_t)h * N + qi] = mt + __log2f(lt);
    const float inv = vsc[2 * slot + 1] / lt;
    const int64_t yo = (qi * H + h) * kD + d0;
    if (ydt == DT_BF16) {
#pragma unroll
        for (int k8 = 0; k8 < 2; ++k8) {
            bf16x8 o;
#pragma unroll
            for (int k = 0; k < 8; ++k) o[k] = (bf16)(acc[8 * k8 + k] * inv);
            *reinterpret_cast<bf16x8*>(reinterpret_cast<bf16*>(Y) + yo + 8 * k8) = o;
        }
    } else {
        float* y = reinterpret_cast<float*>(Y) + yo;
#pragma unroll
        for (int k = 0; k < 4; ++k)
            *reinterpret_cast<float4*>(y + 4 * k) = make_float4(
                acc[4 * k] * inv, acc[4 * k + 1] * inv, acc[4 * k + 2] * inv, acc[4 * k + 3] * inv);
    }
}

// ------------------------------------------------------------------------
// K6b (bf16, wide logit range): one workgroup = 4 waves x 64 queries of one
// FULL head; runs only the work items that K6a flagged.
// Per 64-key tile and wave:  S^T = K Q^T  (keys x queries, 2 x 2 blocks of
// 32x32, 16 MFMAs), online softmax in registers, O^T += V^T P^T (d x queries,
// 16 MFMAs).  Each lane owns one query column of every block, so softmax row
// statistics stay in the lane plus one exchange with lane ^ 32.  K rows are
// stored in LDS with index bits 2 and 3 swapped so that the S^T registers
// hold eight consecutive keys per lane-half: they become the B operand of the
// PV MFMA without any data movement.
//
// Softmax work per score is one FMA, one exp2, half an fp16 pack and half a
// dot2 (row sums of the packed P).  The running maximum m is a reference
// point, not necessarily the exact maximum: a tile whose logits provably stay
// below m + 8 (in log2 units; Cauchy-Schwarz, |q . k| c <= |q| c max|k|) is
// exponentiated against m directly, so p <= 2^8 fits fp16.  Only otherwise is
// the tile maximum computed, and m moves (rescaling O and l) only when the
// tile exceeds m + 8; the key that set m has p = 1, so l >= 1 and weights
// below fp16's normal range add at most 2^-25 each.  O / l is unchanged by
// the choice of reference point.
// ------------------------------------------------------------------------
template <bool kTeach>
__global__ __launch_bounds__(256, 2) void k_flash_bf16_wide(const bf16* __restrict__ Q,
                                                       const bf16* __restrict__ K,
                                                       const f16* __restrict__ Vt,
                                                       const float* __restrict__ kmax,
                                                       const float* __restrict__ vsc,
                                                       const int32_t* __restrict__ buckets,
                                                       int64_t N, int H, int nqt, int nkt, float c,
                                                       const int32_t* __restrict__ wide_items,
                                                       int nqt_fast, void* __restrict__ Y, int ydt,
                                                       float* __restrict__ off) {
    const int nfull = full_count(buckets, H);
    const int active = nfull * nqt;
    if ((int)blockIdx.x >= active) return;
    const int L = xcd_remap(blockIdx.x, active);
    const int slot = L / nqt, qt = L - slot * nqt;
    const int h = full_head(buckets, H, slot);
    if (h < 0 || wide_items[slot * nqt_fast + qt / (kBQf / kBQ16)] == 0) return;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int n = lane & 31, hh = lane >> 5;

    __shared__ __attribute__((aligned(16))) bf16 sK[2][kBK * kLdsRow];
    __shared__ __attribute__((aligned(16))) f16 sV[2][kD * kLdsRow];

    // Q^T operands of this wave's two 32-query blocks, kept in registers,
    // and |q| * c per query for the logit bound.
    bf16x8 Qop[2][4];
    int64_t qidx[2];
    float qnc[2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const int64_t qi = (int64_t)qt * kBQ16 + wave * 64 + qb * 32 + n;
        qidx[qb] = qi;
        const bool ok = qi < N;
        const bf16* qp = Q + ((ok ? qi : 0) * H + h) * kD + 8 * hh;
        float n2 = 0.f;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            Qop[qb][ks] = load_bf16x8(qp + 16 * ks);
            if (!ok) Qop[qb][ks] = zero_bf16x8();
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float x = bf16_to_f32(Qop[qb][ks][j]);
                n2 = fmaf(x, x, n2);
            }
        }
        n2 += __shfl_xor(n2, 32);
        qnc[qb] = sqrtf(n2) * c;
    }

    // Global -> LDS copy assignment: 64 rows x 4 segments of 16 elements.
    const int lr = threadIdx.x >> 2, lc = (threadIdx.x & 3) * 16;
    const f16* Vth = Vt + (int64_t)slot * nkt * kD * kBK;
    const float* kmx = kmax + (int64_t)slot * nkt;
    bf16x8 pk0, pk1;
    f16x8 pv0, pv1;
    // Keys past N read row 0 instead (always in bounds); their logits are
    // masked to -inf in the last tile, so their values never matter.  (No
    // select on the loaded data: it would stall on the prefetch.)
    auto gload = [&](int t) {
        const int64_t key = (int64_t)t * kBK + lr;
        const bf16* kp = K + ((key < N ? key : 0) * H + h) * kD + lc;
        pk0 = load_bf16x8(kp);
        pk1 = load_bf16x8(kp + 8);
        const f16* vp = Vth + ((int64_t)t * kD + lr) * kBK + lc;
        pv0 = *reinterpret_cast<const f16x8*>(vp);
        pv1 = *reinterpret_cast<const f16x8*>(vp + 8);
    };
    auto lstore = [&](int buf) {
        bf16* kd = &sK[buf][swap23(lr) * kLdsRow + lc];
        *reinterpret_cast<bf16x8*>(kd) = pk0;
        *reinterpret_cast<bf16x8*>(kd + 8) = pk1;
        f16* vd = &sV[buf][lr * kLdsRow + lc];
        *reinterpret_cast<f16x8*>(vd) = pv0;
        *reinterpret_cast<f16x8*>(vd + 8) = pv1;
    };

    f32x16 O[2][2];
    float m[2], l[2], le[2];   // le: Kahan compensation of l (teacher instances)
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        O[qb][0] = O[qb][1] = zero_f32x16();
        m[qb] = -INFINITY;
        l[qb] = le[qb] = 0.f;
    }

    gload(0);
    lstore(0);
    __syncthreads();

    for (int t = 0; t < nkt; ++t) {
        const int buf = t & 1;
        const float kbound = kmx[t];
        if (t + 1 < nkt) gload(t + 1);

        // Per 32-query block: S^T = K Q^T, then its probabilities.  Blocks are
        // done one after the other to keep one S^T live (the K operand is
        // re-read from LDS for the second block).
        const bool last = (int64_t)(t + 1) * kBK > N;
        f16x8 P[2][2][2];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            f32x16 S[2];
            S[0] = S[1] = zero_f32x16();
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    const bf16x8 a = *reinterpret_cast<const bf16x8*>(
                        &sK[buf][(kb * 32 + n) * kLdsRow + 16 * ks + 8 * hh]);
                    S[kb] = mfma_bf16(a, Qop[qb][ks], S[kb]);
                }
            if (last) {   // ragged last tile: mask keys >= N
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int64_t key =
                            (int64_t)t * kBK + kb * 32 + 16 * (r >> 3) + 8 * hh + (r & 7);
                        if (key >= N) S[kb][r] = -INFINITY;
                    }
            }
            // Reference point: keep m unless the bound cannot rule out a
            // logit above m + kSlack for some query of this block.
            if (__builtin_amdgcn_ballot_w64(qnc[qb] * kbound > m[qb] + kSlack) != 0) {
                float mx = -INFINITY;
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, S[kb][r]);
                mx = fmaxf(mx, __shfl_xor(mx, 32)) * c;
                const bool move = mx > m[qb] + kSlack;
                const float mn = move ? mx : m[qb];
                const float al = move ? exp2f_fast(m[qb] - mn) : 1.f;
                m[qb] = mn;
                l[qb] *= al;
                le[qb] *= al;
#pragma unroll
                for (int db = 0; db < 2; ++db)
#pragma unroll
                    for (int r = 0; r < 16; ++r) O[qb][db][r] *= al;
            }
            // p = 2^(s c - m), packed to fp16; row sums per tile from zero, then
            // added to l: from the packed values, or in teacher instances from
            // the fp32 values with a compensated add.
            const float nm = -m[qb];
            float ls = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    u32x4 pk;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        f32x2 e;
                        e[0] = exp2f_fast(fmaf(S[kb][8 * b + 2 * j], c, nm));
                        e[1] = exp2f_fast(fmaf(S[kb][8 * b + 2 * j + 1], c, nm));
                        pk[j] = __builtin_bit_cast(uint32_t, __builtin_convertvector(e, f16x2));
                        if (kTeach)
                            ls += e[0] + e[1];
                        else
                            ls = dot2_ones(pk[j], ls);
                    }
                    P[qb][kb][b] = __builtin_bit_cast(f16x8, pk);
                }
            if (kTeach)
                kahan_add(l[qb], le[qb], ls);
            else
                l[qb] += ls;
        }

        // O^T += V^T P^T
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    const f16x8 a = *reinterpret_cast<const f16x8*>(
                        &sV[buf][(db * 32 + n) * kLdsRow + kb * 32 + 16 * b + 8 * hh]);
#pragma unroll
                    for (int qb = 0; qb < 2; ++qb) O[qb][db] = mfma_f16(a, P[qb][kb][b], O[qb][db]);
                }

        if (t + 1 < nkt) lstore(buf ^ 1);
        __syncthreads();
    }

    if (kTeach) {
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) l[qb] -= le[qb];
    }
    store_rows(O, l, qidx, N, H, h, hh, vsc[2 * slot + 1], Y, ydt);
    if (kTeach) store_offsets(l, m, qidx, N, h, hh, off);
}

// ------------------------------------------------------------------------
// K6 (fp32): one workgroup = 4 waves x 32 queries; 32x32x2 fp32 MFMA.  S^T
// output register r of lane-half hh holds key 8 (r / 4) + 4 hh + (r % 4) of
// its 32-key block; the PV MFMA consumes one register per step, reading the
// matching V row from LDS.  Small layers (few work items for the chip) split
// each item's key tiles into two halves run by separate workgroups; each
// half writes O (unnormalized, relative to its reference point m), l and m
// per query, and K6d combines the two halves in order.
// ------------------------------------------------------------------------
constexpr int kBQ32 = 128;
constexpr int kKRow32 = 65;   // odd stride: column reads are bank-conflict free
constexpr int kRec32 = kD + 4;   // split record: O[64], l, m, 2 pad (16-byte aligned)

__global__ __launch_bounds__(256, 2) void k_flash_f32(const float* __restrict__ Q,
                                                      const float* __restrict__ K,
                                                      const float* __restrict__ V,
                                                      const int32_t* __restrict__ buckets,
                                                      int64_t N, int H, int nqt, int nkt, float c,
                                                      int splits, float* __restrict__ part,
                                                      void* __restrict__ Y, int ydt) {
    const int nfull = full_count(buckets, H);
    const int active = nfull * nqt;
    if ((int)blockIdx.x >= active * splits) return;
    const int Lx = xcd_remap(blockIdx.x, active * splits);
    const int L = Lx / splits, half = Lx - L * splits;
    const int slot = L / nqt, qt = L - slot * nqt;
    // key tiles [t0, t1) of the item (all of them unless split)
    const int t0 = (int)((int64_t)half * nkt / splits);
    const int t1 = (int)((int64_t)(half + 1) * nkt / splits);
    const int h = full_head(buckets, H, slot);
    if (h < 0) return;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int n = lane & 31, hh = lane >> 5;

    __shared__ float sK[2][kBK * kKRow32];
    __shared__ __attribute__((aligned(16))) float sV[2][kBK * kD];

    const int64_t qi = (int64_t)qt * kBQ32 + wave * 32 + n;
    const bool qok = qi < N;
    float Qf[32];
    {
        const float* qp = Q + ((qok ? qi : 0) * H + h) * kD + hh;
#pragma unroll
        for (int ks = 0; ks < 32; ++ks) Qf[ks] = qok ? qp[2 * ks] : 0.f;
    }

    const int lr = threadIdx.x >> 2, lc = (threadIdx.x & 3) * 16;
    // Keys past N read row 0 (in bounds); their logits are masked to -inf,
    // so they get weight exactly 0 (inputs are finite).
    float4 pk0, pk1, pk2, pk3, pv0, pv1, pv2, pv3;
    auto gload = [&](int t) {
        const int64_t key = (int64_t)t * kBK + lr;
        const int64_t row = key < N ? key : 0;
        const float4* kp = reinterpret_cast<const float4*>(K + (row * H + h) * kD + lc);
        const float4* vp = reinterpret_cast<const float4*>(V + (row * H + h) * kD + lc);
        pk0 = kp[0]; pk1 = kp[1]; pk2 = kp[2]; pk3 = kp[3];
        pv0 = vp[0]; pv1 = vp[1]; pv2 = vp[2]; pv3 = vp[3];
    };
    auto put4 = [](float* d, float4 v) {
        d[0] = v.x; d[1] = v.y; d[2] = v.z; d[3] = v.w;
    };
    auto lstore = [&](int buf) {
        float* kd = &sK[buf][lr * kKRow32 + lc];
        put4(kd, pk0); put4(kd + 4, pk1); put4(kd + 8, pk2); put4(kd + 12, pk3);
        float4* vd = reinterpret_cast<float4*>(&sV[buf][lr * kD + lc]);
        vd[0] = pv0; vd[1] = pv1; vd[2] = pv2; vd[3] = pv3;
    };

    f32x16 O[2] = {zero_f32x16(), zero_f32x16()};
    float m = -INFINITY, l = 0.f;
    gload(t0);
    lstore(0);
    __syncthreads();

    for (int t = t0; t < t1; ++t) {
        const int buf = (t - t0) & 1;
        if (t + 1 < t1) gload(t + 1);
        f32x16 S[2] = {zero_f32x16(), zero_f32x16()};
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int ks = 0; ks < 32; ++ks)
                S[kb] = mfma_f32(sK[buf][(kb * 32 + n) * kKRow32 + 2 * ks + hh], Qf[ks], S[kb]);
        if ((int64_t)(t + 1) * kBK > N) {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int64_t key = (int64_t)t * kBK + kb * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
                    if (key >= N) S[kb][r] = -INFINITY;
                }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, S[kb][r]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float mn = fmaxf(m, mx * c);
        const float al = exp2f_fast(m - mn);
        m = mn;
        // Two-level sums: the tile's weights and its PV product are summed
        // from zero, then added to the running l and O, so that rounding
        // grows with the tile count rather than the key count.
        float ls = 0.f;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float p = exp2f_fast(fmaf(S[kb][r], c, -mn));
                S[kb][r] = p;
                ls += p;
            }
        l = fmaf(l, al, ls);
        f32x16 Ot[2] = {zero_f32x16(), zero_f32x16()};
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = kb * 32 + 8 * (r >> 2) + 4 * hh + (r & 3);
                    Ot[db] = mfma_f32(sV[buf][key * kD + db * 32 + n], S[kb][r], Ot[db]);
                }
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int r = 0; r < 16; ++r) O[db][r] = fmaf(O[db][r], al, Ot[db][r]);
        if (t + 1 < t1) lstore(buf ^ 1);
        __syncthreads();
    }

    const float lt = l + __shfl_xor(l, 32);
    if (splits > 1) {
        float* pr = part + ((int64_t)(L * 2 + half) * kBQ32 + wave * 32 + n) * kRec32;
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                *reinterpret_cast<float4*>(pr + db * 32 + 8 * g + 4 * hh) =
                    make_float4(O[db][4 * g], O[db][4 * g + 1], O[db][4 * g + 2],
                                O[db][4 * g + 3]);
        if (hh == 0) {
            pr[kD] = lt;
            pr[kD + 1] = m;
        }
        return;
    }
    const float inv = 1.f / lt;
    if (qok) {
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int64_t off = (qi * H + h) * kD + db * 32 + 8 * g + 4 * hh;
                const float y0 = O[db][4 * g] * inv, y1 = O[db][4 * g + 1] * inv;
                const float y2 = O[db][4 * g + 2] * inv, y3 = O[db][4 * g + 3] * inv;
                if (ydt == DT_BF16) {
                    bf16x4 v;
                    v[0] = (bf16)y0; v[1] = (bf16)y1; v[2] = (bf16)y2; v[3] = (bf16)y3;
                    *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(Y) + off) = v;
                } else {
                    *reinterpret_cast<float4*>(reinterpret_cast<float*>(Y) + off) =
                        make_float4(y0, y1, y2, y3);
                }
            }
    }
}

// K6d: Y of the fp32 items that K6 split into two key halves: the halves' O
// and l scaled to the larger reference point and added (half 0, then half
// 1), then O / l.  Two workgroups of 256 threads per item, 4 threads per
// query and 16 of its values each.
__global__ __launch_bounds__(256) void k_flash_f32_combine(const int32_t* __restrict__ buckets,
                                                           int64_t N, int H, int nqt,
                                                           const float* __restrict__ part,
                                                           void* __restrict__ Y, int ydt) {
    const int nfull = full_count(buckets, H);
    const int L = blockIdx.x >> 1;
    if (L >= nfull * nqt) return;
    const int slot = L / nqt, qt = L - slot * nqt;
    const int h = full_head(buckets, H, slot);
    if (h < 0) return;
    const int qr = (blockIdx.x & 1) * 64 + (threadIdx.x >> 2), d0 = (threadIdx.x & 3) * 16;
    const int64_t qi = (int64_t)qt * kBQ32 + qr;
    if (qi >= N) return;
    const float* r0 = part + ((int64_t)(L * 2) * kBQ32 + qr) * kRec32;
    const float* r1 = r0 + (int64_t)kBQ32 * kRec32;
    const float m0 = r0[kD + 1], m1 = r1[kD + 1];
    const float mt = fmaxf(m0, m1);
    const float w0 = exp2f_fast(m0 - mt), w1 = exp2f_fast(m1 - mt);
    const float inv = 1.f / fmaf(r1[kD], w1, r0[kD] * w0);
    float y[16];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const float4 a = *reinterpret_cast<const float4*>(r0 + d0 + 4 * k);
        const float4 b = *reinterpret_cast<const float4*>(r1 + d0 + 4 * k);
        y[4 * k] = fmaf(b.x, w1, a.x * w0) * inv;
        y[4 * k + 1] = fmaf(b.y, w1, a.y * w0) * inv;
        y[4 * k + 2] = fmaf(b.z, w1, a.z * w0) * inv;
        y[4 * k + 3] = fmaf(b.w, w1, a.w * w0) * inv;
    }
    const int64_t yo = (qi * H + h) * kD + d0;
    if (ydt == DT_BF16) {
#pragma unroll
        for (int k8 = 0; k8 < 2; ++k8) {
            bf16x8 o;
#pragma unroll
            for (int k = 0; k < 8; ++k) o[k] = (bf16)y[8 * k8 + k];
            *reinterpret_cast<bf16x8*>(reinterpret_cast<bf16*>(Y) + yo + 8 * k8) = o;
        }
    } else {
        float* yp = reinterpret_cast<float*>(Y) + yo;
#pragma unroll
        for (int k = 0; k < 4; ++k)
            *reinterpret_cast<float4*>(yp + 4 * k) =
                make_float4(y[4 * k], y[4 * k + 1], y[4 * k + 2], y[4 * k + 3]);
    }
}

// ------------------------------------------------------------------ launchers

int flash_q_tile(int dtype) { return dtype == DT_BF16 ? kBQ16 : kBQ32; }

int flash_stream_groups(int64_t N, int H) {
    (void)N;
    (void)H;
    return kStreamWG;
}

size_t flash_part_bytes(int64_t N, int H) {
    return (size_t)2 * flash_stream_groups(N, H) * kPartFloats * sizeof(float);
}

// fp32 layers: two key halves per work item while the items alone would
// leave the chip short of waves (at most 2 workgroups per CU of them), and
// the workspace for the halves' records.
int flash_f32_splits(int64_t N, int H) {
    const int64_t nqt = (N + kBQ32 - 1) / kBQ32, nkt = (N + kBK - 1) / kBK;
    return nqt * H <= 2 * kStreamWG && nkt >= 2 ? 2 : 1;
}
size_t flash_f32_part_bytes(int64_t N, int H) {
    if (flash_f32_splits(N, H) == 1) return 0;
    const int64_t nqt = (N + kBQ32 - 1) / kBQ32;
    return (size_t)H * nqt * 2 * kBQ32 * kRec32 * sizeof(float);
}

int64_t flash_vmax_parts(int64_t N) {
    const int64_t nkt = (N + kBK - 1) / kBK;
    return (nkt + kVmaxTiles - 1) / kVmaxTiles;
}

void launch_gather(const AttnArgs& a, hipStream_t st) {
    const int nkt = (int)((a.N + kBK - 1) / kBK);
    const int nvp = (int)flash_vmax_parts(a.N);
    hipLaunchKernelGGL(k_vmax_partial, dim3(nvp, a.H), dim3(256), 0, st, (const bf16*)a.V,
                       a.buckets, a.N, a.H, a.vpart);
    hipLaunchKernelGGL(k_gather_vt, dim3(nkt, a.H), dim3(256), 0, st, (const bf16*)a.K,
                       (const bf16*)a.V, a.buckets, a.N, a.H, nkt, (const float*)a.vpart, nvp,
                       a.vsc, (f16*)a.vt, (f16*)a.kh, a.kmax);
}

void launch_flash(const AttnArgs& a, hipStream_t st) {
    const int nkt = (int)((a.N + kBK - 1) / kBK);
    const float c = kLog2e / sqrtf((float)kD);
    const int bq = flash_q_tile(a.dtype);
    const int nqt = (int)((a.N + bq - 1) / bq);
    if (a.dtype == DT_BF16) {
        const int nqf = (int)((a.N + kBQf - 1) / kBQf);
        const int G = flash_stream_groups(a.N, a.H);
        hipLaunchKernelGGL(a.off ? k_flash_bf16<true> : k_flash_bf16<false>, dim3(G), dim3(512),
                           0, st, (const bf16*)a.Q, (const f16*)a.kh, (const f16*)a.vt,
                           (const float*)a.kmax, (const float*)a.vsc, a.buckets, a.N, a.H, nqf,
                           nkt, c, a.qflag, a.part, G, a.Y, a.ydt, a.off);
        hipLaunchKernelGGL(k_flash_combine, dim3(G * (kBQf / kCombRows)), dim3(256), 0, st,
                           a.buckets, a.N, a.H, nqf,
                           nkt, (const int32_t*)a.qflag, (const float*)a.part,
                           (const float*)a.vsc, G, a.Y, a.ydt, a.off);
        hipLaunchKernelGGL(a.off ? k_flash_bf16_wide<true> : k_flash_bf16_wide<false>,
                           dim3(nqt * a.H), dim3(256), 0, st, (const bf16*)a.Q, (const bf16*)a.K,
                           (const f16*)a.vt, (const float*)a.kmax, (const float*)a.vsc, a.buckets,
                           a.N, a.H, nqt, nkt, c, a.qflag, nqf, a.Y, a.ydt, a.off);
    } else {
        const int splits = flash_f32_splits(a.N, a.H);
        hipLaunchKernelGGL(k_flash_f32, dim3(nqt * a.H * splits), dim3(256), 0, st,
                           (const float*)a.Q, (const float*)a.K, (const float*)a.V, a.buckets,
                           a.N, a.H, nqt, nkt, c, splits, a.part, a.Y, a.ydt);
        if (splits > 1)
            hipLaunchKernelGGL(k_flash_f32_combine, dim3(nqt * a.H * 2), dim3(256), 0, st,
                               a.buckets, a.N, a.H, nqt, (const float*)a.part, a.Y, a.ydt);
    }
}

}  // namespace vp
