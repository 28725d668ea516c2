// The dense block around the routed layer (Algorithm 1, steps 1, 3 and 4):
//   X~ = LN_1(X);  (Q, K, V) = QKV(X~) with the 2D rotary encoding of the
//   token positions applied to Q and K;  [routed attention: Y];
//   X_attn = X + LS_1 (Y W_O^T + b_O);
//   X_out  = X_attn + LS_2 (W_fc2 GELU(W_fc1 LN_2(X_attn) + b_fc1) + b_fc2).
// Two kinds of kernel: a LayerNorm (one wave per row, HBM-bound) and a bf16
// GEMM on MFMA whose epilogue applies the bias and then the step's own
// elementwise work (rotary encoding and the split into Q, K, V; GELU; or
// LayerScale plus residuals), so no projection output makes an extra trip
// through HBM.  The residual stream is never rounded in between: the W_O
// step stores only the attention update A = LS_1 (Y W_O^T + b_O), and LN_2
// and the last step form X_attn = X + A in fp32 from X and A.
#include "vp_device.hpp"
#include "vp_internal.hpp"

namespace vp {

constexpr int kDm = 1024;   // model width D = 16 heads x 64

// ------------------------------------------------------------------------
// B1: LayerNorm over the D = 1024 features of each row of X (+ X2 when given,
// added in fp32): mean and biased variance in fp32 (two passes over
// registers), y = (x - mean) r g + b, r = 1 / sqrt(var + eps), rounded to
// bf16.  One wave per kLnRows consecutive rows, g and b held in registers;
// lane l holds features 8 l ... 8 l + 7 and 512 + 8 l ... 512 + 8 l + 7, so
// each 16-byte load or store of a wave covers 1 KB of the row contiguously.
// The next row's loads are issued before the current row is normalised.
// ------------------------------------------------------------------------
constexpr int kLnRows = 2;

template <bool kAdd>
__global__ __launch_bounds__(256) void k_layernorm(const bf16* __restrict__ X,
                                                   const bf16* __restrict__ X2, int64_t T,
                                                   const float* __restrict__ g,
                                                   const float* __restrict__ b, float eps,
                                                   bf16* __restrict__ Y) {
    const int64_t row0 =
        ((int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6)) * kLnRows;
    if (row0 >= T) return;
    const int lane = threadIdx.x & 63, c0 = 8 * lane, c1 = kDm / 2 + 8 * lane;
    float gg[16], bv[16];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        gg[j] = g[c0 + j];
        gg[8 + j] = g[c1 + j];
        bv[j] = b[c0 + j];
        bv[8 + j] = b[c1 + j];
    }
    const int nr = T - row0 < kLnRows ? (int)(T - row0) : kLnRows;
    constexpr int kV = kAdd ? 4 : 2;
    auto load = [&](int64_t row, bf16x8 (&v)[kV]) {
        const bf16* xr = X + row * kDm;
        v[0] = load_bf16x8(xr + c0);
        v[1] = load_bf16x8(xr + c1);
        if constexpr (kAdd) {
            const bf16* x2 = X2 + row * kDm;
            v[2] = load_bf16x8(x2 + c0);
            v[3] = load_bf16x8(x2 + c1);
        }
    };
    auto norm = [&](int64_t row, const bf16x8 (&v)[kV]) {
        float x[16];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            x[j] = bf16_to_f32(v[0][j]);
            x[8 + j] = bf16_to_f32(v[1][j]);
            if constexpr (kAdd) {
                x[j] += bf16_to_f32(v[2][j]);
                x[8 + j] += bf16_to_f32(v[3][j]);
            }
        }
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < 16; ++j) s += x[j];
        const float mean = wave_sum(s) * (1.f / kDm);
        float q = 0.f;
#pragma unroll
        for (int j = 0; j < 16; ++j) q = fmaf(x[j] - mean, x[j] - mean, q);
        const float r = rsqrtf(wave_sum(q) * (1.f / kDm) + eps);
        float y[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) y[j] = fmaf((x[j] - mean) * r, gg[j], bv[j]);
        bf16* yr = Y + row * kDm;
        *reinterpret_cast<bf16x8*>(yr + c0) =
            pack_bf16x8(y[0], y[1], y[2], y[3], y[4], y[5], y[6], y[7]);
        *reinterpret_cast<bf16x8*>(yr + c1) =
            pack_bf16x8(y[8], y[9], y[10], y[11], y[12], y[13], y[14], y[15]);
    };
    // Straight-line over kLnRows rows with two register sets, each row's loads
    // issued one row ahead of its use.  Rows past the last are the last row
    // again (the same values stored twice; Y never aliases X or X2), so no
    // branch sits around the loads and each wait covers only the row in use.
    auto rowi = [&](int i) { return row0 + (i < nr ? i : nr - 1); };
    bf16x8 v[2][kV];
    load(rowi(0), v[0]);
#pragma unroll
    for (int i = 0; i < kLnRows; ++i) {
        if (i + 1 < kLnRows) load(rowi(i + 1), v[(i + 1) & 1]);
        __builtin_amdgcn_sched_barrier(0);  // keep the prefetch ahead of the row's arithmetic
        norm(rowi(i), v[i & 1]);
    }
}

// ------------------------------------------------------------------------
// B2: D^T = W X^T for W [F, Kd] (weights as stored, [out, in]) and X [T, Kd]
// (token rows), bf16 operands, fp32 accumulation: both operands are
// Kd-contiguous, as the MFMA wants them.  Workgroup tile 256 features x 256
// tokens, Kd in stages of 64 through two LDS buffers (144-byte rows:
// conflict-free 16-byte reads).  Output features are the MFMA rows, so lane l
// holds token l % 32 of a block and features 8 (r / 4) + 4 (l / 32) + r % 4 in
// its register r: four consecutive features per store, and the rotary pair
// (j, j + 16) of a 32-feature half in registers r and r + 8 of one lane.
// Tiles are ordered with all of a token tile's feature tiles together, and
// consecutive tiles share an XCD, so an XCD's L2 keeps a token tile for all
// its feature tiles while the weights stream by.
// Every output sums its Kd products in the same order (stage by stage, 16 per
// MFMA) in both kernels below, so they produce identical bits.
// ------------------------------------------------------------------------
constexpr int kGM = 256, kGN = 256, kGK = 64, kGRow = 72;
constexpr int kGemmWG = 256;   // persistent workgroups: one per CU

// EPI_RESID: ls (acc + bias) + res + res2, either residual may be null;
// EPI_RESID2: the same with both residuals given.
enum { EPI_QKV = 0, EPI_GELU = 1, EPI_RESID = 2, EPI_RESID2 = 3 };

struct GemmArgs {
    const bf16* W;        // [F, Kd]
    const bf16* X;        // [T, Kd]
    const float* bias;    // [F]
    int64_t T;
    int F, Kd;
    bf16* out;            // GELU, RESID, RESID2: [T, F]
    const bf16 *res, *res2;   // RESID: residuals [T, F] (either may be null); RESID2: both
    const float* ls;      // RESID, RESID2: LayerScale [F]
    bf16 *q, *k, *v;      // QKV: [T, D] each
    const int32_t* pos;   // QKV: [T, 2] (row, column)
    float log2_base;      // QKV: log2 of the rotary base
};

// Tile (L) of the grouped order, `group` feature tiles per token tile:
// features f0.., tokens t0...
__device__ __forceinline__ void gemm_tile(int L, int ntt, int group, int& f0, int64_t& t0) {
    const int grp = L / (group * ntt), in = L - grp * group * ntt;
    const int tt = in / group, ft = grp * group + in % group;
    f0 = ft * kGM;
    t0 = (int64_t)tt * kGN;
}

// Epilogue of a wave's 128 features x (32 NTB) tokens: lane (n, hh) holds, in
// acc[fb][tb] register r = 4 gq + i, feature f0 + 128 wm + 32 fb + 8 gq + 4 hh
// + i of token tl + tok0 + 32 tb + n.  Tokens outside [t0, T) are not stored.
template <int EPI, int NTB>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& g, f32x16 (&acc)[4][NTB], int f0,
                                              int64_t t0, int64_t tl, int wm, int tok0, int n,
                                              int hh, const float* sbl = nullptr) {
    float omega[8];   // rotary frequencies of features j = 8 (r / 4) + 4 hh + r % 4, r < 8
    if (EPI == EPI_QKV) {
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const int j = 8 * (r >> 2) + 4 * hh + (r & 3);
            omega[r] = exp2f(-(float)j * (1.f / 16.f) * g.log2_base);
        }
    }
    // All of a wave's features lie in one of Q, K, V (f0 is a multiple of
    // 256); Q and K are rotated, the first 32 features of each 64 by the row
    // coordinate and the next 32 by the column coordinate.
    const bool rotate = EPI == EPI_QKV && (f0 + 128 * wm) / kDm < 2;
    // The 8-wave kernel (NTB = 2) reads the wave's 64 bias values once, with
    // one wait, for all its tokens; the persistent kernel, whose registers are
    // full, reads the tile's bias and LayerScale from LDS (sbl: 256 bias values,
    // then 256 LayerScale values, for features f0 ...) per 32 x 32 block.
    constexpr bool kHoist = NTB == 2;
    float bias[4][16];
    if constexpr (kHoist) {
#pragma unroll
        for (int fb = 0; fb < 4; ++fb)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                bias[fb][r] = g.bias[f0 + 128 * wm + 32 * fb + 8 * (r >> 2) + 4 * hh + (r & 3)];
    }
    // The wave's output tensor, chosen once with a wave-uniform index (an index
    // in vector registers made the compiler read the pointer from the
    // argument block per 32 x 32 block and wait for it before each store).
    const int which = EPI == EPI_QKV ? __builtin_amdgcn_readfirstlane((f0 + 128 * wm) / kDm) : 0;
    bf16* const qkv_out = which == 0 ? g.q : (which == 1 ? g.k : g.v);
    // Rotary positions of all the wave's tokens, read before the first is
    // used (rows past T - 1 read row T - 1 and are not stored).
    int2 pos[NTB];
    if (rotate) {
#pragma unroll
        for (int tb = 0; tb < NTB; ++tb) {
            const int64_t t = tl + tok0 + 32 * tb + n;
            pos[tb] = *reinterpret_cast<const int2*>(g.pos + 2 * (t < g.T ? t : g.T - 1));
        }
    }
#pragma unroll
    for (int tb = 0; tb < NTB; ++tb) {
        const int64_t t = tl + tok0 + 32 * tb + n;
        if (t < t0 || t >= g.T) continue;
        // An offset the compiler cannot see through, so the LDS reads of
        // bias and LayerScale stay in each block instead of being hoisted out
        // of the token loop (128 values per lane held across it spill).
        int lo = -f0;
        if (sbl) asm volatile("" : "+v"(lo));
        // (sin, cos) of this token's angles, once per token: half 0 takes the
        // row coordinate, half 1 the column coordinate
        float rs[2][8], rc[2][8];
        if (rotate) {
            const int2 p = pos[tb];
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                __sincosf((float)p.x * omega[r], &rs[0][r], &rc[0][r]);
                __sincosf((float)p.y * omega[r], &rs[1][r], &rc[1][r]);
            }
        }
#pragma unroll
        for (int fb = 0; fb < 4; ++fb) {
            const int fbase = f0 + 128 * wm + 32 * fb;
            float v[16];
#pragma unroll
            for (int r = 0; r < 16; ++r)
                v[r] = acc[fb][tb][r] +
                       (kHoist ? bias[fb][r]
                               : sbl ? sbl[fbase + lo + 8 * (r >> 2) + 4 * hh + (r & 3)]
                                     : g.bias[fbase + 8 * (r >> 2) + 4 * hh + (r & 3)]);
            bf16* dst;
            if (EPI == EPI_QKV) {
                const int fin = fbase - which * kDm;
                if (rotate) {   // Q, K: rotate the planes (j, j + 16) of this half
                    const int half = (fin & 32) ? 1 : 0;   // fb & 1
#pragma unroll
                    for (int r = 0; r < 8; ++r) {
                        const float sn = rs[half][r], cs = rc[half][r];
                        const float u = v[r], w = v[r + 8];
                        v[r] = u * cs - w * sn;
                        v[r + 8] = u * sn + w * cs;
                    }
                }
                dst = qkv_out + t * kDm + fin;
            } else {
                dst = g.out + t * g.F + fbase;
                if (EPI == EPI_GELU) {
#pragma unroll
                    for (int r = 0; r < 16; ++r) v[r] = gelu(v[r]);
                } else if (EPI == EPI_RESID2) {   // ls (acc + bias) + res + res2, in fp32
                    // Both residuals are read with no branch around the loads,
                    // so the reads of the four feature groups are in flight
                    // together (a null test per read waits for each one).
                    float base[16];
#pragma unroll
                    for (int gq = 0; gq < 4; ++gq) {
                        const int f = fbase + 8 * gq + 4 * hh;
                        const bf16x4 r1 = *reinterpret_cast<const bf16x4*>(g.res + t * g.F + f);
                        const bf16x4 r2 = *reinterpret_cast<const bf16x4*>(g.res2 + t * g.F + f);
#pragma unroll
                        for (int i = 0; i < 4; ++i) base[4 * gq + i] = (float)r1[i] + (float)r2[i];
                    }
#pragma unroll
                    for (int gq = 0; gq < 4; ++gq) {
                        const int f = fbase + 8 * gq + 4 * hh;
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            v[4 * gq + i] = fmaf(sbl ? sbl[kGM + f + lo + i] : g.ls[f + i],
                                                 v[4 * gq + i], base[4 * gq + i]);
                    }
                } else {   // ls (acc + bias) + res + res2, summed in fp32
#pragma unroll
                    for (int gq = 0; gq < 4; ++gq) {
                        const int f = fbase + 8 * gq + 4 * hh;
                        float base[4] = {0.f, 0.f, 0.f, 0.f};
                        if (g.res) {
                            const bf16x4 rs = *reinterpret_cast<const bf16x4*>(g.res + t * g.F + f);
#pragma unroll
                            for (int i = 0; i < 4; ++i) base[i] = (float)rs[i];
                        }
                        if (g.res2) {
                            const bf16x4 rs = *reinterpret_cast<const bf16x4*>(g.res2 + t * g.F + f);
#pragma unroll
                            for (int i = 0; i < 4; ++i) base[i] += (float)rs[i];
                        }
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            v[4 * gq + i] = fmaf(sbl ? sbl[kGM + f + lo + i] : g.ls[f + i],
                                                 v[4 * gq + i], base[i]);
                    }
                }
            }
#pragma unroll
            for (int gq = 0; gq < 4; ++gq) {
                bf16x4 o;
#pragma unroll
                for (int i = 0; i < 4; ++i) o[i] = (bf16)v[4 * gq + i];
                *reinterpret_cast<bf16x4*>(dst + 8 * gq + 4 * hh) = o;
            }
        }
    }
}

// B2a (W_O and FFN 2 projections, T >= 256): persistent, one workgroup of 4
// waves per CU, each wave a 128 x 128 block of the tile with its 256
// accumulators in AGPRs.  Workgroup b
// takes tiles i G + slot(b), slot grouping the workgroups of an XCD, so the 32
// tiles an XCD runs at once are 8 token tiles x 4 feature tiles.  A partial
// last token tile reads rows T - 256 .. T - 1 (every read in bounds) and
// stores only its own tokens.
// Pipeline: stage s + 2 is loaded into registers while stage s is multiplied
// (two register sets, so two stages are in flight), stage s + 1 goes to LDS
// during the last k-step of stage s, and the next tile's first stages are in
// flight during a tile's epilogue.  Per stage a wave issues 64 MFMAs
// (4 k-steps x 16), 32 LDS fragment reads (each k-step reads the next one's),
// 16 global loads and 16 LDS stores, interleaved one for one with the MFMAs
// by scheduling barriers; the one barrier per stage sits between the two
// halves of the last k-step, whose second half covers the first reads of the
// next stage.
template <int EPI>
__global__ __launch_bounds__(256, 1) void k_gemm(GemmArgs g) {
    // Make the AGPRs available to the register allocator (accumulators).
    asm volatile("" ::: "a0");
    const int nft = g.F / kGM;
    const int ntt = (int)((g.T + kGN - 1) / kGN);
    const int total = nft * ntt;
    const int nk = g.Kd / kGK;
    const int G = gridDim.x, b = blockIdx.x;
    const int slot = (G & 7) == 0 ? (b & 7) * (G >> 3) + (b >> 3) : b;
    const int ntile = slot < total ? (total - 1 - slot) / G + 1 : 0;
    if (ntile == 0) return;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int n = lane & 31, hh = lane >> 5;
    const int wm = wave >> 1, wn = wave & 1;

    __shared__ __attribute__((aligned(16))) bf16 sW[2][kGM * kGRow];
    __shared__ __attribute__((aligned(16))) bf16 sX[2][kGN * kGRow];
    __shared__ __attribute__((aligned(16))) float sBL[2 * kGM];   // the tile's bias, LayerScale

    // All of a token tile's feature tiles in one group (with FFN 1 on this
    // kernel, 16 feature tiles, so that an XCD's 32 tiles were 2 token tiles
    // x 16 feature tiles, were 3 % faster than groups of 4; 2.6 % on QKV in
    // B2b).
    auto tile_of = [&](int i, int& f0, int64_t& t0, int64_t& tl) {
        gemm_tile(i * G + slot, ntt, nft, f0, t0);
        tl = t0 + kGN <= g.T ? t0 : g.T - kGN;
    };

    // Load state: the next stage to load (tile li, stage lkt).  Past the last
    // stage the bases keep pointing at a valid stage; those loads go unused.
    int li = 0, lkt = 0, lf0;
    int64_t lt0, ltl;
    tile_of(0, lf0, lt0, ltl);
    const char* wb;
    const char* xb;
    auto next_bases = [&]() {
        wb = reinterpret_cast<const char*>(g.W + (int64_t)lf0 * g.Kd + lkt * kGK);
        xb = reinterpret_cast<const char*>(g.X + ltl * g.Kd + lkt * kGK);
        if (++lkt == nk) {
            lkt = 0;
            if (++li < ntile) tile_of(li, lf0, lt0, ltl);
        }
    };
    // Thread tid moves row (tid / 8) + 32 j, bytes 16 (tid % 8) of the
    // stage's 128, j = 0..7, of both operands.
    const uint32_t voff = (uint32_t)(tid >> 3) * (uint32_t)g.Kd * 2u + (uint32_t)(tid & 7) * 16u;
    const int64_t jstride = (int64_t)32 * g.Kd * 2;
    auto gload = [&](int h, u32x4 (&rw)[8], u32x4 (&rx)[8]) {
#pragma unroll
        for (int j = 4 * h; j < 4 * h + 4; ++j) {
            rw[j] = *reinterpret_cast<const u32x4*>(wb + j * jstride + voff);
            rx[j] = *reinterpret_cast<const u32x4*>(xb + j * jstride + voff);
        }
    };
    const int lsoff = (tid >> 3) * kGRow + (tid & 7) * 8;
    auto lstore = [&](int buf, u32x4 (&rw)[8], u32x4 (&rx)[8]) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            *reinterpret_cast<u32x4*>(&sW[buf][lsoff + 32 * j * kGRow]) = rw[j];
            *reinterpret_cast<u32x4*>(&sX[buf][lsoff + 32 * j * kGRow]) = rx[j];
        }
    };
    const int aoff = (128 * wm + n) * kGRow + 8 * hh, xoff = (128 * wn + n) * kGRow + 8 * hh;
    auto lread = [&](int buf, int ks, bf16x8 (&a)[4], bf16x8 (&x)[4]) {
#pragma unroll
        for (int fb = 0; fb < 4; ++fb)
            a[fb] = *reinterpret_cast<const bf16x8*>(&sW[buf][aoff + 32 * fb * kGRow + 16 * ks]);
#pragma unroll
        for (int tb = 0; tb < 4; ++tb)
            x[tb] = *reinterpret_cast<const bf16x8*>(&sX[buf][xoff + 32 * tb * kGRow + 16 * ks]);
    };

    f32x16 acc[4][4];
#pragma unroll
    for (int fb = 0; fb < 4; ++fb)
#pragma unroll
        for (int tb = 0; tb < 4; ++tb) acc[fb][tb] = zero_f32x16();

    u32x4 ra[8], xa[8], rb[8], xb8[8];   // the two register sets
    next_bases();
    gload(0, ra, xa);
    gload(1, ra, xa);
    next_bases();
    gload(0, rb, xb8);
    gload(1, rb, xb8);
    lstore(0, ra, xa);
    __syncthreads();
    bf16x8 fa0[4], fx0[4], fa1[4], fx1[4];
    lread(0, 0, fa0, fx0);
    int buf = 0;

#define VP_SGB(mask, cnt) __builtin_amdgcn_sched_group_barrier(mask, cnt, 0)
#define VP_MMA(A, X, FB0, FB1)                                                          \
    _Pragma("unroll") for (int fb = FB0; fb < FB1; ++fb)                               \
        _Pragma("unroll") for (int tb = 0; tb < 4; ++tb) acc[fb][tb] =                  \
            mfma_bf16(A[fb], X[tb], acc[fb][tb]);
    // One stage: load the stage after next into (LW, LX), store the next
    // stage from (SW, SX).  Masks: 0x008 MFMA, 0x020 global load, 0x100 LDS
    // read, 0x200 LDS write.
#define VP_STAGE(LW, LX, SW, SX)                                                        \
    {                                                                                   \
        next_bases();                                                                   \
        lread(buf, 1, fa1, fx1);                                                        \
        gload(0, LW, LX);                                                               \
        VP_MMA(fa0, fx0, 0, 4);                                                         \
        for (int q = 0; q < 8; ++q) { VP_SGB(0x008, 1); VP_SGB(0x100, 1); VP_SGB(0x020, 1); } \
        VP_SGB(0x008, 8);                                                               \
        lread(buf, 2, fa0, fx0);                                                        \
        gload(1, LW, LX);                                                               \
        VP_MMA(fa1, fx1, 0, 4);                                                         \
        for (int q = 0; q < 8; ++q) { VP_SGB(0x008, 1); VP_SGB(0x100, 1); VP_SGB(0x020, 1); } \
        VP_SGB(0x008, 8);                                                               \
        lread(buf, 3, fa1, fx1);                                                        \
        VP_MMA(fa0, fx0, 0, 4);                                                         \
        for (int q = 0; q < 8; ++q) { VP_SGB(0x008, 1); VP_SGB(0x100, 1); }             \
        VP_SGB(0x008, 8);                                                               \
        VP_MMA(fa1, fx1, 0, 2);                                                         \
        lstore(buf ^ 1, SW, SX);                                                        \
        for (int q = 0; q < 8; ++q) { VP_SGB(0x008, 1); VP_SGB(0x200, 2); }             \
        __syncthreads();                                                                \
        lread(buf ^ 1, 0, fa0, fx0);                                                    \
        VP_MMA(fa1, fx1, 2, 4);                                                         \
        for (int q = 0; q < 8; ++q) { VP_SGB(0x008, 1); VP_SGB(0x100, 1); }             \
        buf ^= 1;                                                                       \
    }
    for (int i = 0; i < ntile; ++i) {
        for (int kt = 0; kt < nk; kt += 2) {   // nk is even
            VP_STAGE(ra, xa, rb, xb8);
            VP_STAGE(rb, xb8, ra, xa);
        }
        int f0;
        int64_t t0, tl;
        tile_of(i, f0, t0, tl);
        // The tile's bias and LayerScale through LDS: one read and one wait per
        // thread, then one barrier, instead of a read and a wait per 32 x 32
        // block.  The previous tile's epilogue finished reading sBL before the
        // barriers of this tile's stages.
        sBL[tid] = g.bias[f0 + tid];
        sBL[kGM + tid] = g.ls[f0 + tid];
        __syncthreads();
        gemm_epilogue<EPI, 4>(g, acc, f0, t0, tl, wm, 128 * wn, n, hh, sBL);
#pragma unroll
        for (int fb = 0; fb < 4; ++fb)
#pragma unroll
            for (int tb = 0; tb < 4; ++tb) acc[fb][tb] = zero_f32x16();
    }
#undef VP_STAGE
#undef VP_MMA
#undef VP_SGB
}

// B2b: one workgroup per tile, 8 waves of 128 x 64 (two per SIMD), the stage
// copy through registers one stage ahead, token rows past T reading row T - 1
// (their outputs are never stored).  Used for the QKV projection, whose
// rotary epilogue (16 sincos per token) the second wave on each SIMD helps
// to hide (3-8 % faster than B2a at S = 100), for FFN 1, whose GELU epilogue
// it hides likewise (output stage 1 % faster), and for T < 256.
template <int EPI>
__global__ __launch_bounds__(512, 1) void k_gemm_w8(GemmArgs g) {
    const int nft = g.F / kGM;
    const int ntt = (int)((g.T + kGN - 1) / kGN);
    const int total = nft * ntt;
    int f0;
    int64_t t0;
    gemm_tile(xcd_remap(blockIdx.x, total), ntt, nft, f0, t0);
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int n = lane & 31, hh = lane >> 5;
    const int wm = wave >> 2, wn = wave & 3;

    __shared__ __attribute__((aligned(16))) bf16 sW[2][kGM * kGRow];
    __shared__ __attribute__((aligned(16))) bf16 sX[2][kGN * kGRow];

    // Stage copy: 4 chunks of 16 bytes of W and 4 of X per thread; chunk
    // c = tid + 512 i is row c / 8, bytes 16 (c % 8) of the stage's 128.
    u32x4 rw[4], rx[4];
    auto gload = [&](int kt) {
        const int k0 = kt * kGK;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = tid + 512 * i, row = c >> 3, seg = (c & 7) * 8;
            rw[i] = *reinterpret_cast<const u32x4*>(g.W + (int64_t)(f0 + row) * g.Kd + k0 + seg);
            const int64_t tr = t0 + row < g.T ? t0 + row : g.T - 1;
            rx[i] = *reinterpret_cast<const u32x4*>(g.X + tr * g.Kd + k0 + seg);
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = tid + 512 * i, row = c >> 3, seg = (c & 7) * 8;
            *reinterpret_cast<u32x4*>(&sW[buf][row * kGRow + seg]) = rw[i];
            *reinterpret_cast<u32x4*>(&sX[buf][row * kGRow + seg]) = rx[i];
        }
    };

    f32x16 acc[4][2];
#pragma unroll
    for (int fb = 0; fb < 4; ++fb) acc[fb][0] = acc[fb][1] = zero_f32x16();

    gload(0);
    lstore(0);
    __syncthreads();
    const int nk = g.Kd / kGK;
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
        for (int ks = 0; ks < kGK / 16; ++ks) {
            bf16x8 a[4], x[2];
#pragma unroll
            for (int fb = 0; fb < 4; ++fb)
                a[fb] = *reinterpret_cast<const bf16x8*>(
                    &sW[buf][(128 * wm + 32 * fb + n) * kGRow + 16 * ks + 8 * hh]);
#pragma unroll
            for (int tb = 0; tb < 2; ++tb)
                x[tb] = *reinterpret_cast<const bf16x8*>(
                    &sX[buf][(64 * wn + 32 * tb + n) * kGRow + 16 * ks + 8 * hh]);
#pragma unroll
            for (int fb = 0; fb < 4; ++fb)
#pragma unroll
                for (int tb = 0; tb < 2; ++tb) acc[fb][tb] = mfma_bf16(a[fb], x[tb], acc[fb][tb]);
        }
        if (kt + 1 < nk) lstore(buf ^ 1);
        __syncthreads();
    }
    gemm_epilogue<EPI, 2>(g, acc, f0, t0, t0, wm, 64 * wn, n, hh);
}

// ------------------------------------------------------------------ launchers

template <int EPI>
static void gemm_launch(const GemmArgs& a, hipStream_t st) {
    const int total = (a.F / kGM) * (int)((a.T + kGN - 1) / kGN);
    if constexpr (EPI == EPI_RESID || EPI == EPI_RESID2) {
        if (a.T >= kGN) {
            hipLaunchKernelGGL(k_gemm<EPI>, dim3(total < kGemmWG ? total : kGemmWG), dim3(256), 0,
                               st, a);
            return;
        }
    }
    hipLaunchKernelGGL(k_gemm_w8<EPI>, dim3(total), dim3(512), 0, st, a);
}

// F a multiple of 256, Kd of 128 (the persistent kernel takes stages in
// pairs); the block's shapes are 1024 x
// {3, 1, 4} by 1024 and 1024 by 4096.
static void gemm(int epi, const GemmArgs& a, hipStream_t st) {
    if (epi == EPI_QKV)
        gemm_launch<EPI_QKV>(a, st);
    else if (epi == EPI_GELU)
        gemm_launch<EPI_GELU>(a, st);
    else if (epi == EPI_RESID2 && a.res && a.res2)
        gemm_launch<EPI_RESID2>(a, st);
    else
        gemm_launch<EPI_RESID>(a, st);
}

static void layernorm(const bf16* X, const bf16* X2, int64_t T, const float* g, const float* b,
                      float eps, bf16* Y, hipStream_t st) {
    const dim3 grid((unsigned)((T + 4 * kLnRows - 1) / (4 * kLnRows)));
    if (X2)
        hipLaunchKernelGGL(k_layernorm<true>, grid, dim3(256), 0, st, X, X2, T, g, b, eps, Y);
    else
        hipLaunchKernelGGL(k_layernorm<false>, grid, dim3(256), 0, st, X, X2, T, g, b, eps, Y);
}

void launch_block_qkv(const BlockArgs& a, hipStream_t st) {
    layernorm(a.X, nullptr, a.T, a.ln1_w, a.ln1_b, a.eps, a.ln, st);
    GemmArgs g = {};
    g.W = a.w_qkv; g.X = a.ln; g.bias = a.b_qkv; g.T = a.T; g.F = 3 * kDm; g.Kd = kDm;
    g.q = a.Q; g.k = a.K; g.v = a.V; g.pos = a.pos; g.log2_base = log2f(a.rope_base);
    gemm(EPI_QKV, g, st);
}

void launch_block_out(const BlockArgs& a, hipStream_t st) {
    GemmArgs g = {};
    g.T = a.T;
    // A = LS_1 (Y W_O^T + b_O), the attention update (X_attn = X + A)
    g.W = a.w_o; g.X = a.Y; g.bias = a.b_o; g.F = kDm; g.Kd = kDm;
    g.res = nullptr; g.res2 = nullptr; g.ls = a.ls1; g.out = a.xa;
    gemm(EPI_RESID, g, st);
    layernorm(a.X, a.xa, a.T, a.ln2_w, a.ln2_b, a.eps, a.ln, st);
    // H = GELU(LN_2(X + A) W_fc1^T + b_fc1)
    g.W = a.w_fc1; g.X = a.ln; g.bias = a.b_fc1; g.F = 4 * kDm; g.Kd = kDm; g.out = a.hid;
    gemm(EPI_GELU, g, st);
    // X_out = X + A + LS_2 (H W_fc2^T + b_fc2)
    g.W = a.w_fc2; g.X = a.hid; g.bias = a.b_fc2; g.F = kDm; g.Kd = 4 * kDm;
    g.res = a.X; g.res2 = a.xa; g.ls = a.ls2; g.out = a.Xout;
    gemm(EPI_RESID2, g, st);
}

}  // namespace vp
