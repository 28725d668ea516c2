// The two linear-cost modes of the routed layer:
//   SURR (Section 4.3, Eq.5-7): y_i = C_h + gamma_i (.) delta_i with
//        gamma_i = sigmoid(MLP_gamma([v_i; C_h])), delta_i = MLP_delta([v_i; C_h]);
//   MEAN (Algorithm 1, third branch): y_i = (1/N) sum_j v_j for every token.
// and the ablations of SURR that Section 5.3 evaluates (Tables 5-6): the
// value mean as context, no residual correction (y_i = C_h), the identity
// added (y_i = v_i + Eq.7) and linear attention in place of the surrogate.
// Each kernel runs over (token block, head) and exits unless modes[h] is its
// mode.
//
// The first MLP layer splits z = [v; C] into W1 = [W1_v | W1_C]: the context
// half W1_C C_h + b1 is the same for every token of a head and is computed
// once per workgroup, leaving a 64 x 64 product per token.
#include "vp_device.hpp"
#include "vp_internal.hpp"

namespace vp {

__device__ __forceinline__ float act_fn(float x, int act) {
    if (act == 1) return fmaxf(x, 0.f);
    return gelu(x);
}

__device__ __forceinline__ float sigmoid_fast(float x) {
    return rcp_fast(1.f + exp2f_fast(-kLog2e * x));
}

// Tokens per workgroup: 384 (fewer weight copies per token), down to 128
// when that would leave fewer than kSurrMinGroups workgroups over all heads.
constexpr int kSurrRows = 384;
constexpr int kSurrMinGroups = 2048;
constexpr int kW = 72;           // bf16 LDS row stride

// ------------------------------------------------------------------------
// K7 (bf16): per wave and 32 tokens, H1^T = W1_v V^T (128 x 32: rows 0-63
// gamma hidden, 64-127 delta hidden; 16 MFMAs), activation, then
// G^T = W2_gamma H_gamma^T and D^T = W2_delta H_delta^T (64 x 32 each,
// 8 MFMAs each).  W1 rows sit in LDS with index bits 2,3 swapped so that
// hidden units arrive eight-consecutive per lane-half, the K order of the
// second MFMA.
// ------------------------------------------------------------------------
// kAddV: the identity added (y = v + Eq.7), an instance of its own so that
// the Eq.7 instance carries none of its registers.
template <int ACT, bool kAddV>
__global__ __launch_bounds__(256, 4) void k_surrogate_bf16(
    const bf16* __restrict__ V, const uint8_t* __restrict__ modes, const float* __restrict__ ctx,
    const bf16* __restrict__ gw1, const float* __restrict__ gb1, const bf16* __restrict__ gw2,
    const float* __restrict__ gb2, const bf16* __restrict__ dw1, const float* __restrict__ db1,
    const bf16* __restrict__ dw2, const float* __restrict__ db2, int64_t N, int H,
    int rows, void* __restrict__ Y, int ydt) {
    const int h = blockIdx.y;
    if (modes[h] != MODE_SURR) return;
    const int64_t t0 = (int64_t)blockIdx.x * rows;
    const int64_t t1 = (t0 + rows < N) ? t0 + rows : N;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int n = lane & 31, hh = lane >> 5;

    __shared__ __attribute__((aligned(16))) bf16 sW1[128 * kW];   // [hidden (permuted)][d]
    __shared__ __attribute__((aligned(16))) bf16 sW2[2][64 * kW]; // [gamma|delta][d][hidden]
    __shared__ __attribute__((aligned(16))) float sC[kD], sB2g[kD], sB2d[kD], sC1[128];

    const float* C = ctx + h * kD;
    if (tid < kD) {
        sC[tid] = C[tid];
        sB2g[tid] = gb2[h * kD + tid];
        sB2d[tid] = db2[h * kD + tid];
    }
    // Context half of layer 1 plus bias: c1[u] = b1[u] + sum_c W1[u][64 + c] C[c],
    // summed in c order.  Threads 0..127 load their row's 64 weights now and
    // sum once C is in LDS.
    bf16x8 wc[8];
    float c1acc = 0.f;
    if (tid < 128) {
        const int u = tid & 63;
        const bf16* w1 = (tid < 64 ? gw1 : dw1) + ((int64_t)h * kL + u) * 2 * kD + kD;
#pragma unroll
        for (int k = 0; k < 8; ++k) wc[k] = load_bf16x8(w1 + 8 * k);
        c1acc = (tid < 64 ? gb1 : db1)[h * kL + u];
    }
    // W1_v rows (value half) into LDS, rows permuted within 32-blocks.
    for (int i = tid; i < 128 * 8; i += 256) {
        const int u = i >> 3, seg = (i & 7) * 8;
        const bf16* w1 = (u < 64 ? gw1 : dw1) + ((int64_t)h * kL + (u & 63)) * 2 * kD + seg;
        *reinterpret_cast<bf16x8*>(&sW1[swap23(u & 31) * kW + (u & ~31) * kW + seg]) =
            load_bf16x8(w1);
    }
    for (int i = tid; i < 2 * 64 * 8; i += 256) {
        const int which = i >> 9, r = (i >> 3) & 63, seg = (i & 7) * 8;
        const bf16* w2 = (which == 0 ? gw2 : dw2) + ((int64_t)h * kD + r) * kL + seg;
        *reinterpret_cast<bf16x8*>(&sW2[which][r * kW + seg]) = load_bf16x8(w2);
    }
    __syncthreads();
    if (tid < 128) {
#pragma unroll
        for (int cc = 0; cc < kD; ++cc) c1acc = fmaf(bf16_to_f32(wc[cc >> 3][cc & 7]), sC[cc], c1acc);
        sC1[tid] = c1acc;
    }
    __syncthreads();


    // Each wave takes 32 tokens at a time; the next block's V is loaded while
    // this one is computed.  Tokens past t1 read token t0 (never stored).
    auto load_v = [&](int64_t tb, bf16x8 (&B)[4]) {
        const int64_t tok = tb + n;
        const bf16* vr = V + ((tok < t1 ? tok : t0) * H + h) * kD + 8 * hh;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) B[ks] = load_bf16x8(vr + 16 * ks);
    };
    bf16x8 B[4], Bn[4];
    load_v(t0 + 32 * wave, B);
    for (int64_t tb = t0 + 32 * wave; tb < t1; tb += 128) {
        const int64_t tok = tb + n;
        const bool ok = tok < t1;
        load_v(tb + 128 < t1 ? tb + 128 : tb, Bn);
        // One MLP at a time (gamma: hidden blocks 0, 1 and W2_gamma; delta:
        // blocks 2, 3 and W2_delta), so only one MLP's hidden layer is live.
        // The weight fragments are read from LDS every iteration (an opaque
        // offset keeps them from being hoisted into 128 loop-long registers,
        // which would leave room for one wave per SIMD).
        int wrow = n * kW + 8 * hh;
        asm volatile("" : "+v"(wrow));
        f32x16 G[2], D[2];
#pragma unroll
        for (int which = 0; which < 2; ++which) {
            f32x16 A1[2];
#pragma unroll
            for (int m2 = 0; m2 < 2; ++m2) {
                const int mb = 2 * which + m2;
                A1[m2] = zero_f32x16();
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    const bf16x8 a = *reinterpret_cast<const bf16x8*>(
                        &sW1[32 * mb * kW + wrow + 16 * ks]);
                    A1[m2] = mfma_bf16(a, B[ks], A1[m2]);
                }
            }
            bf16x8 Hop[4];   // k-steps over this MLP's 64 hidden units
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                // register r0 + j of block mb holds hidden unit 32 mb + 16 (ks % 2) + 8 hh + j
                const int m2 = ks >> 1, mb = 2 * which + m2, r0 = 8 * (ks & 1);
                const f32x4 ca = *reinterpret_cast<const f32x4*>(&sC1[32 * mb + 2 * r0 + 8 * hh]);
                const f32x4 cb = *reinterpret_cast<const f32x4*>(&sC1[32 * mb + 2 * r0 + 8 * hh + 4]);
                float hv[8];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    hv[j] = act_fn(A1[m2][r0 + j] + ca[j], ACT);
                    hv[4 + j] = act_fn(A1[m2][r0 + 4 + j] + cb[j], ACT);
                }
                Hop[ks] = pack_bf16x8(hv[0], hv[1], hv[2], hv[3], hv[4], hv[5], hv[6], hv[7]);
            }
#pragma unroll
            for (int db = 0; db < 2; ++db) {
                f32x16 o = zero_f32x16();
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    const bf16x8 aw = *reinterpret_cast<const bf16x8*>(
                        &sW2[which][32 * db * kW + wrow + 16 * ks]);
                    o = mfma_bf16(aw, Hop[ks], o);
                }
                if (which == 0) G[db] = o; else D[db] = o;
            }
        }
        if (ok) {
            // The token's 8 value groups, read together before the first is
            // used (one wait, not one per group).
            bf16x4 vin[2][4];
            if constexpr (kAddV) {
#pragma unroll
                for (int db = 0; db < 2; ++db)
#pragma unroll
                    for (int g = 0; g < 4; ++g)
                        vin[db][g] = *reinterpret_cast<const bf16x4*>(
                            V + (tok * H + h) * kD + 32 * db + 8 * g + 4 * hh);
            }
#pragma unroll
            for (int db = 0; db < 2; ++db)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int d0 = 32 * db + 8 * g + 4 * hh;
                    float y[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int d = d0 + i;
                        const float gam = sigmoid_fast(G[db][4 * g + i] + sB2g[d]);
                        y[i] = sC[d] + gam * (D[db][4 * g + i] + sB2d[d]);
                    }
                    const int64_t off = (tok * H + h) * kD + d0;
                    if constexpr (kAddV) {   // identity added: y = v + Eq.7
#pragma unroll
                        for (int i = 0; i < 4; ++i) y[i] += (float)vin[db][g][i];
                    }
                    if (ydt == DT_BF16) {
                        bf16x4 v;
                        v[0] = (bf16)y[0]; v[1] = (bf16)y[1]; v[2] = (bf16)y[2]; v[3] = (bf16)y[3];
                        *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(Y) + off) = v;
                    } else {
                        *reinterpret_cast<float4*>(reinterpret_cast<float*>(Y) + off) =
                            make_float4(y[0], y[1], y[2], y[3]);
                    }
                }
        }
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) B[ks] = Bn[ks];
    }
}

// ------------------------------------------------------------------------
// K7 (fp32): the same two-layer MLP on fp32 32x32x2 MFMAs; a wave takes 32
// tokens (lane l: token l % 32, half hh = l / 32), a workgroup 128.
//   layer 1: H1^T = W1_v V^T + (W1_C C_h + b1)   (128 hidden x 32 tokens,
//            4 blocks x 32 steps); step s reduces over value features s
//            (lanes hh = 0) and 32 + s (hh = 1), so a lane holds one
//            contiguous half of its token's value row;
//   layer 2: G^T = W2_gamma act(H1_gamma)^T, D^T = W2_delta act(H1_delta)^T
//            (64 x 32 each); step s of hidden block ub reduces over the two
//            hidden units that layer 1's output register s holds in the two
//            lane halves (8 (s / 4) + 4 hh + s % 4), so those registers are
//            the B operand as they are.
// W1's value half sits in LDS row-major with stride 65 floats, W2 transposed
// ([hidden][d]) with stride 72: both MFMA A-operand reads are bank-conflict
// free.
// ------------------------------------------------------------------------
constexpr int kSurr32Rows = 128;   // tokens per workgroup (4 waves x 32)
constexpr int kW1s = 65, kW2s = 72;

template <int ACT>
__global__ __launch_bounds__(256, 2) void k_surrogate_f32(
    const float* __restrict__ V, const uint8_t* __restrict__ modes, const float* __restrict__ ctx,
    const float* __restrict__ gw1, const float* __restrict__ gb1, const float* __restrict__ gw2,
    const float* __restrict__ gb2, const float* __restrict__ dw1, const float* __restrict__ db1,
    const float* __restrict__ dw2, const float* __restrict__ db2, int add_v, int64_t N, int H,
    void* __restrict__ Y, int ydt) {
    const int h = blockIdx.y;
    if (modes[h] != MODE_SURR) return;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, n = lane & 31, hh = lane >> 5;
    __shared__ float sW1[2 * kL * kW1s];        // [gamma units | delta units][value feature]
    __shared__ float sW2t[2][kL * kW2s];        // [which][hidden][d]
    __shared__ float sC1[2 * kL], sC[kD], sB2[2][kD];
    const float* C = ctx + h * kD;
    for (int i = tid; i < 2 * kL * kD; i += 256) {
        const int u = i / kD, c = i % kD;        // unit u of [gamma | delta], feature c
        const float* w1 = (u < kL ? gw1 : dw1) + ((int64_t)h * kL + (u & (kL - 1))) * 2 * kD;
        sW1[u * kW1s + c] = w1[c];
        const int which = u / kL, uu = u % kL;   // here (uu, c) = (d, hidden) of W2
        const float* w2 = (which == 0 ? gw2 : dw2) + (int64_t)h * kD * kL;
        sW2t[which][c * kW2s + uu] = w2[uu * kL + c];
    }
    if (tid < 2 * kL) {
        const int which = tid / kL, u = tid % kL;
        const float* w1 = (which == 0 ? gw1 : dw1) + ((int64_t)h * kL + u) * 2 * kD;
        float acc = (which == 0 ? gb1 : db1)[h * kL + u];
        for (int c = 0; c < kD; ++c) acc = fmaf(w1[kD + c], C[c], acc);
        sC1[tid] = acc;
    }
    if (tid < kD) {
        sC[tid] = C[tid];
        sB2[0][tid] = gb2[h * kD + tid];
        sB2[1][tid] = db2[h * kD + tid];
    }
    __syncthreads();

    const int64_t tok = (int64_t)blockIdx.x * kSurr32Rows + wave * 32 + n;
    const bool ok = tok < N;
    float v[32];
    {
        const float4* vr = reinterpret_cast<const float4*>(V + ((ok ? tok : 0) * H + h) * kD + 32 * hh);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const float4 x = ok ? vr[q] : make_float4(0.f, 0.f, 0.f, 0.f);
            v[4 * q] = x.x; v[4 * q + 1] = x.y; v[4 * q + 2] = x.z; v[4 * q + 3] = x.w;
        }
    }
    // Layer 1: block ub holds hidden units 32 ub + 8 (r / 4) + 4 hh + r % 4 in
    // register r; the accumulators start at the per-head constant W1_C C_h + b1.
    f32x16 acc[4];
#pragma unroll
    for (int ub = 0; ub < 4; ++ub)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[ub][r] = sC1[32 * ub + 8 * (r >> 2) + 4 * hh + (r & 3)];
#pragma unroll
    for (int st = 0; st < 32; ++st)
#pragma unroll
        for (int ub = 0; ub < 4; ++ub)
            acc[ub] = mfma_f32(sW1[(32 * ub + n) * kW1s + 32 * hh + st], v[st], acc[ub]);
#pragma unroll
    for (int ub = 0; ub < 4; ++ub)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            acc[ub][r] = ACT == 1 ? fmaxf(acc[ub][r], 0.f) : gelu_erf(acc[ub][r]);
    // Layer 2: output block db holds d = 32 db + 8 (r / 4) + 4 hh + r % 4.
    f32x16 og[2], od[2];
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int d = 32 * db + 8 * (r >> 2) + 4 * hh + (r & 3);
            og[db][r] = sB2[0][d];
            od[db][r] = sB2[1][d];
        }
#pragma unroll
    for (int ub = 0; ub < 2; ++ub)
#pragma unroll
        for (int st = 0; st < 16; ++st) {
            const int u = 32 * ub + 8 * (st >> 2) + 4 * hh + (st & 3);
#pragma unroll
            for (int db = 0; db < 2; ++db) {
                og[db] = mfma_f32(sW2t[0][u * kW2s + 32 * db + n], acc[ub][st], og[db]);
                od[db] = mfma_f32(sW2t[1][u * kW2s + 32 * db + n], acc[2 + ub][st], od[db]);
            }
        }
    if (!ok) return;
    const int64_t row = (tok * H + h) * kD;
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int d0 = 32 * db + 8 * q + 4 * hh;
            float y[4];
            float4 vv = make_float4(0.f, 0.f, 0.f, 0.f);
            if (add_v) vv = *reinterpret_cast<const float4*>(V + row + d0);
            const float va[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
            for (int j = 0; j < 4; ++j)
                y[j] = sC[d0 + j] + sigmoid_fast(og[db][4 * q + j]) * od[db][4 * q + j] + va[j];
            if (ydt == DT_BF16) {
                bf16x4 o;
                o[0] = (bf16)y[0]; o[1] = (bf16)y[1]; o[2] = (bf16)y[2]; o[3] = (bf16)y[3];
                *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(Y) + row + d0) = o;
            } else {
                *reinterpret_cast<float4*>(reinterpret_cast<float*>(Y) + row + d0) =
                    make_float4(y[0], y[1], y[2], y[3]);
            }
        }
}

// ------------------------------------------------------------------------
// K8: a write-only stream of one [d] vector per head into every row: MEAN
// heads (the value mean) and SURR heads of the no-residual ablation (C_h).
// 8 lanes per row (8 values each); a workgroup covers 32 rows per step.
// ------------------------------------------------------------------------
constexpr int kMeanRows = 1024;

__global__ __launch_bounds__(256) void k_broadcast_heads(const uint8_t* __restrict__ modes,
                                                         int mode, const float* __restrict__ vmean,
                                                         int64_t N, int H, void* __restrict__ Y,
                                                         int ydt) {
    const int h = blockIdx.y;
    if (modes[h] != mode) return;
    const int64_t t0 = (int64_t)blockIdx.x * kMeanRows;
    const int64_t t1 = (t0 + kMeanRows < N) ? t0 + kMeanRows : N;
    const int seg = (threadIdx.x & 7) * 8, rr = threadIdx.x >> 3;
    float mv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) mv[j] = vmean[h * kD + seg + j];
    if (ydt == DT_BF16) {
        const bf16x8 v = pack_bf16x8(mv[0], mv[1], mv[2], mv[3], mv[4], mv[5], mv[6], mv[7]);
        for (int64_t row = t0 + rr; row < t1; row += 32)
            *reinterpret_cast<bf16x8*>(reinterpret_cast<bf16*>(Y) + (row * H + h) * kD + seg) = v;
    } else {
        const float4 a = make_float4(mv[0], mv[1], mv[2], mv[3]);
        const float4 b = make_float4(mv[4], mv[5], mv[6], mv[7]);
        for (int64_t row = t0 + rr; row < t1; row += 32) {
            float4* p = reinterpret_cast<float4*>(reinterpret_cast<float*>(Y) + (row * H + h) * kD + seg);
            p[0] = a;
            p[1] = b;
        }
    }
}

// ------------------------------------------------------------------------
// Linear attention in place of the surrogate (compute-mode ablation,
// Table 6; Katharopoulos et al.), non-causal over all N tokens with
// phi(x) = elu(x) + 1:  y_i = phi(q_i)^T S / phi(q_i) . z with
// S = sum_j phi(k_j) v_j^T (64 x 64) and z = sum_j phi(k_j).
// Both contractions run on the fp32 MFMA (32x32x2: exact fp32 products,
// operands taken straight from the row-major [N, H, 64] rows), sums in fp32:
//   K10a  per (token chunk, head): partial S and z of the chunk;
//   K10b  per head: S and z summed over the chunks in chunk order;
//   K10c  per (32-query block, head): y_i.
// ------------------------------------------------------------------------
__device__ __forceinline__ float elu1(float x) {
    return x > 0.f ? x + 1.f : exp2f_fast(x * kLog2e);
}

// Elements 2c and 2c + 1 of the 64-value row starting at element `off`.
template <int DT>
__device__ __forceinline__ float2 load_pair(const void* __restrict__ X, int64_t off, int c) {
    if (DT == DT_BF16) {
        const uint32_t w = *reinterpret_cast<const uint32_t*>(
            reinterpret_cast<const bf16*>(X) + off + 2 * c);
        const bf16x2 v = __builtin_bit_cast(bf16x2, w);
        return make_float2(bf16_to_f32(v[0]), bf16_to_f32(v[1]));
    }
    return *reinterpret_cast<const float2*>(reinterpret_cast<const float*>(X) + off + 2 * c);
}

// 32 consecutive values of a row, as fp32.
template <int DT>
__device__ __forceinline__ void load32(const void* __restrict__ X, int64_t off, float* o) {
    if (DT == DT_BF16) {
        const bf16* p = reinterpret_cast<const bf16*>(X) + off;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const bf16x8 v = load_bf16x8(p + 8 * k);
#pragma unroll
            for (int j = 0; j < 8; ++j) o[8 * k + j] = bf16_to_f32(v[j]);
        }
    } else {
        const float4* p = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(X) + off);
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const float4 v = p[k];
            o[4 * k] = v.x; o[4 * k + 1] = v.y; o[4 * k + 2] = v.z; o[4 * k + 3] = v.w;
        }
    }
}

// K10a.  S^T blocks on MFMA with the token pair as the reduction index:
// A[m][k] = phi(k_{t+k})[2m + mb], B[k][n] = v_{t+k}[2n + nb], so that a lane
// reads one 4-byte pair per row and 32 lanes one whole 128-byte row.  Block
// (mb, nb) register r of lane l then holds S[2m + mb][2n + nb] with
// n = l % 32, m = 8 (r / 4) + 4 (l / 32) + r % 4.  Wave w takes token pairs
// w, w + 4, ..., four per step with the next step's rows already loading; the
// four waves' sums meet in one 16 KB LDS buffer, added in wave order.
template <int DT>
__global__ __launch_bounds__(256) void k_linattn_partial(const void* __restrict__ K,
                                                         const void* __restrict__ V,
                                                         const uint8_t* __restrict__ modes,
                                                         int64_t N, int H, int64_t chunk,
                                                         float* __restrict__ part) {
    const int h = blockIdx.y, c = blockIdx.x;
    if (modes[h] != MODE_SURR) return;
    const int64_t t0 = (int64_t)c * chunk;
    const int64_t t1 = (t0 + chunk < N) ? t0 + chunk : N;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int n = lane & 31, hh = lane >> 5;
    f32x16 acc[2][2];
    float zacc[2] = {0.f, 0.f};
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) acc[mb][0] = acc[mb][1] = zero_f32x16();
    // Rows of step tg: pairs tg + 8 u, u < kLinPairs (wave w starts at
    // t0 + 2 w).
    constexpr int kLinPairs = 4;
    float2 a[kLinPairs], b[kLinPairs], an[kLinPairs], bn[kLinPairs];
    auto load = [&](int64_t tg, float2 (&ka)[kLinPairs], float2 (&vb)[kLinPairs]) {
#pragma unroll
        for (int u = 0; u < kLinPairs; ++u) {
            const int64_t tok = tg + 8 * u + hh;
            ka[u] = vb[u] = make_float2(0.f, 0.f);
            if (tok < t1) {
                const int64_t off = (tok * H + h) * kD;
                ka[u] = load_pair<DT>(K, off, n);
                vb[u] = load_pair<DT>(V, off, n);
            }
        }
    };
    int64_t tg = t0 + 2 * wave;
    load(tg, an, bn);
    for (; tg < t1; tg += 8 * kLinPairs) {
#pragma unroll
        for (int u = 0; u < kLinPairs; ++u) {
            a[u] = an[u];
            b[u] = bn[u];
        }
        if (tg + 8 * kLinPairs < t1) load(tg + 8 * kLinPairs, an, bn);
#pragma unroll
        for (int u = 0; u < kLinPairs; ++u) {
            if (tg + 8 * u + hh < t1) {
                a[u].x = elu1(a[u].x);
                a[u].y = elu1(a[u].y);
            }
            zacc[0] += a[u].x;
            zacc[1] += a[u].y;
            acc[0][0] = mfma_f32(a[u].x, b[u].x, acc[0][0]);
            acc[0][1] = mfma_f32(a[u].x, b[u].y, acc[0][1]);
            acc[1][0] = mfma_f32(a[u].y, b[u].x, acc[1][0]);
            acc[1][1] = mfma_f32(a[u].y, b[u].y, acc[1][1]);
        }
    }
    __shared__ float sP[kD * kD + kD];   // S then z
#pragma unroll 1
    for (int wv = 0; wv < 4; ++wv) {
        if (wave == wv) {
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int m = 8 * (r >> 2) + 4 * hh + (r & 3);
                        float* d = &sP[(2 * m + mb) * kD + 2 * n + nb];
                        *d = wv == 0 ? acc[mb][nb][r] : *d + acc[mb][nb][r];
                    }
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) {
                const float zt = zacc[mb] + __shfl_xor(zacc[mb], 32);
                if (hh == 0) {
                    float* d = &sP[kD * kD + 2 * n + mb];
                    *d = wv == 0 ? zt : *d + zt;
                }
            }
        }
        __syncthreads();
    }
    float* o = part + ((int64_t)h * gridDim.x + c) * kLinSums;
    for (int e = threadIdx.x; e < kLinSums; e += 256) o[e] = sP[e];
}

// K10b.  Grid (cdiv(kLinSums, 256), H): one sum per thread, chunks in order.
__global__ __launch_bounds__(256) void k_linattn_combine(const uint8_t* __restrict__ modes,
                                                         const float* __restrict__ part,
                                                         int nchunks, float* __restrict__ sums) {
    const int h = blockIdx.y;
    if (modes[h] != MODE_SURR) return;
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= kLinSums) return;
    const float* p = part + (int64_t)h * nchunks * kLinSums + i;
    float acc = 0.f;
    for (int c = 0; c < nchunks; ++c) acc += p[(int64_t)c * kLinSums];
    sums[h * kLinSums + i] = acc;
}

// K10c.  Y^T = S^T phi(Q)^T per 32-query block on MFMA: reduction step s
// covers features s and s + 32 (k = l / 32 picks one), so lane l needs the
// contiguous half-row [32 (l / 32), 32 (l / 32) + 32) of its query l % 32,
// and A[m][k] = S[s + 32 k][32 db + m] stays in registers for every block.
// The denominator phi(q) . z is a dot product on the same halves plus one
// exchange with lane l ^ 32.  Each wave takes kLinQBlocks blocks of 32
// queries.
constexpr int kLinQBlocks = 4;

template <int DT>
__global__ __launch_bounds__(256) void k_linattn_apply(const void* __restrict__ Q,
                                                       const uint8_t* __restrict__ modes,
                                                       const float* __restrict__ sums, int64_t N,
                                                       int H, void* __restrict__ Y, int ydt) {
    const int h = blockIdx.y;
    if (modes[h] != MODE_SURR) return;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int n = lane & 31, hh = lane >> 5;
    __shared__ float S[kLinSums];   // the head's S and z, staged once
    for (int i = threadIdx.x; i < kLinSums; i += 256) S[i] = sums[h * kLinSums + i];
    __syncthreads();
    float As[2][32], zr[32];
#pragma unroll
    for (int s = 0; s < 32; ++s) {
        const int dk = s + 32 * hh;
        As[0][s] = S[dk * kD + n];
        As[1][s] = S[dk * kD + 32 + n];
        zr[s] = S[kD * kD + dk];
    }
    // Blocks of this wave: q0(qb) = 32 (first + qb); the next block's
    // half-rows load while the current block's MFMAs run.
    const int64_t first = (int64_t)blockIdx.x * 4 * kLinQBlocks + wave * kLinQBlocks;
    auto qrow = [&](int qb) {
        const int64_t q0 = (first + qb) * 32, qi = q0 + n;
        return ((qi < N ? qi : q0) * H + h) * kD + 32 * hh;
    };
    float fn[32];
    if (first * 32 < N) load32<DT>(Q, qrow(0), fn);
    for (int qb = 0; qb < kLinQBlocks; ++qb) {
        const int64_t q0 = (first + qb) * 32;
        if (q0 >= N) break;
        const int64_t qi = q0 + n;
        const bool ok = qi < N;
        float fq[32];
#pragma unroll
        for (int s = 0; s < 32; ++s) fq[s] = fn[s];
        if (qb + 1 < kLinQBlocks && q0 + 32 < N) load32<DT>(Q, qrow(qb + 1), fn);
        float den = 0.f;
#pragma unroll
        for (int s = 0; s < 32; ++s) {
            fq[s] = elu1(fq[s]);
            den = fmaf(fq[s], zr[s], den);
        }
        den += __shfl_xor(den, 32);
        f32x16 y[2] = {zero_f32x16(), zero_f32x16()};
#pragma unroll
        for (int s = 0; s < 32; ++s) {
            y[0] = mfma_f32(As[0][s], fq[s], y[0]);
            y[1] = mfma_f32(As[1][s], fq[s], y[1]);
        }
        if (ok) {
            const float inv = 1.f / den;
#pragma unroll
            for (int db = 0; db < 2; ++db)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int64_t off = (qi * H + h) * kD + 32 * db + 8 * g + 4 * hh;
                    const float y0 = y[db][4 * g] * inv, y1 = y[db][4 * g + 1] * inv;
                    const float y2 = y[db][4 * g + 2] * inv, y3 = y[db][4 * g + 3] * inv;
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

// ------------------------------------------------------------------ launchers

void launch_linear_heads(const AttnArgs& a, hipStream_t st) {
    int rows = kSurrRows;
    while (rows > 128 && (a.N + rows - 1) / rows * a.H < kSurrMinGroups) rows -= 128;
    const unsigned nbs = (unsigned)((a.N + rows - 1) / rows);
    const int v = a.variant;
    if (v == SURR_EQ7 || v == SURR_MEAN_CONTEXT || v == SURR_ADD_IDENTITY) {
        const float* C = v == SURR_MEAN_CONTEXT ? a.vmean : a.ctx;
        const int add_v = v == SURR_ADD_IDENTITY;
        if (a.dtype == DT_BF16)
        {
            auto* kern = add_v ? (a.act == 1 ? k_surrogate_bf16<1, true> : k_surrogate_bf16<0, true>)
                               : (a.act == 1 ? k_surrogate_bf16<1, false> : k_surrogate_bf16<0, false>);
            hipLaunchKernelGGL(kern, dim3(nbs, a.H), dim3(256), 0, st, (const bf16*)a.V, a.modes, C,
                               (const bf16*)a.g_w1, a.g_b1, (const bf16*)a.g_w2, a.g_b2,
                               (const bf16*)a.d_w1, a.d_b1, (const bf16*)a.d_w2, a.d_b2,
                               a.N, a.H, rows, a.Y, a.ydt);
        }
        else {
            const unsigned nb32 = (unsigned)((a.N + kSurr32Rows - 1) / kSurr32Rows);
            auto* kern = a.act == 1 ? k_surrogate_f32<1> : k_surrogate_f32<0>;
            hipLaunchKernelGGL(kern, dim3(nb32, a.H), dim3(256), 0, st, (const float*)a.V,
                               a.modes, C, (const float*)a.g_w1, a.g_b1, (const float*)a.g_w2,
                               a.g_b2, (const float*)a.d_w1, a.d_b1, (const float*)a.d_w2,
                               a.d_b2, add_v, a.N, a.H, a.Y, a.ydt);
        }
    } else if (v == SURR_NO_RESIDUAL) {
        const unsigned nb = (unsigned)((a.N + kMeanRows - 1) / kMeanRows);
        hipLaunchKernelGGL(k_broadcast_heads, dim3(nb, a.H), dim3(256), 0, st, a.modes,
                           (int)MODE_SURR, a.ctx, a.N, a.H, a.Y, a.ydt);
    } else {   // SURR_LINEAR_ATTN
        const dim3 gp((unsigned)a.n3, a.H), gc((kLinSums + 255) / 256, a.H),
            ga((unsigned)((a.N + 32 * 4 * kLinQBlocks - 1) / (32 * 4 * kLinQBlocks)), a.H);
        if (a.dtype == DT_BF16) {
            hipLaunchKernelGGL(k_linattn_partial<DT_BF16>, gp, dim3(256), 0, st, a.K, a.V,
                               a.modes, a.N, a.H, a.chunk3, a.lpart);
            hipLaunchKernelGGL(k_linattn_combine, gc, dim3(256), 0, st, a.modes, a.lpart,
                               (int)a.n3, a.lsum);
            hipLaunchKernelGGL(k_linattn_apply<DT_BF16>, ga, dim3(256), 0, st, a.Q, a.modes,
                               a.lsum, a.N, a.H, a.Y, a.ydt);
        } else {
            hipLaunchKernelGGL(k_linattn_partial<DT_F32>, gp, dim3(256), 0, st, a.K, a.V,
                               a.modes, a.N, a.H, a.chunk3, a.lpart);
            hipLaunchKernelGGL(k_linattn_combine, gc, dim3(256), 0, st, a.modes, a.lpart,
                               (int)a.n3, a.lsum);
            hipLaunchKernelGGL(k_linattn_apply<DT_F32>, ga, dim3(256), 0, st, a.Q, a.modes,
                               a.lsum, a.N, a.H, a.Y, a.ydt);
        }
    }
    const unsigned nbm = (unsigned)((a.N + kMeanRows - 1) / kMeanRows);
    hipLaunchKernelGGL(k_broadcast_heads, dim3(nbm, a.H), dim3(256), 0, st, a.modes,
                       (int)MODE_MEAN, a.vmean, a.N, a.H, a.Y, a.ydt);
}

}  // namespace vp
