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
    return 0.5f * x * (1.f + erff(x * 0.70710678118654752f));
}

__device__ __forceinline__ float sigmoid_fast(float x) {
    return rcp_fast(1.f + exp2f_fast(-kLog2e * x));
}

constexpr int kSurrRows = 512;   // tokens per workgroup
constexpr int kW = 72;           // bf16 LDS row stride

// ------------------------------------------------------------------------
// K7 (bf16): per wave and 32 tokens, H1^T = W1_v V^T (128 x 32: rows 0-63
// gamma hidden, 64-127 delta hidden; 16 MFMAs), activation, then
// G^T = W2_gamma H_gamma^T and D^T = W2_delta H_delta^T (64 x 32 each,
// 8 MFMAs each).  W1 rows sit in LDS with index bits 2,3 swapped so that
// hidden units arrive eight-consecutive per lane-half, the K order of the
// second MFMA.
// ------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_surrogate_bf16(
    const bf16* __restrict__ V, const uint8_t* __restrict__ modes, const float* __restrict__ ctx,
    const bf16* __restrict__ gw1, const float* __restrict__ gb1, const bf16* __restrict__ gw2,
    const float* __restrict__ gb2, const bf16* __restrict__ dw1, const float* __restrict__ db1,
    const bf16* __restrict__ dw2, const float* __restrict__ db2, int act, int add_v, int64_t N,
    int H, void* __restrict__ Y, int ydt) {
    const int h = blockIdx.y;
    if (modes[h] != MODE_SURR) return;
    const int64_t t0 = (int64_t)blockIdx.x * kSurrRows;
    const int64_t t1 = (t0 + kSurrRows < N) ? t0 + kSurrRows : N;
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
    // Context half of layer 1 plus bias: c1[u] = b1[u] + sum_c W1[u][64 + c] C[c].
    if (tid < 128) {
        const int u = tid & 63;
        const bf16* w1 = (tid < 64 ? gw1 : dw1) + ((int64_t)h * kL + u) * 2 * kD;
        float acc = (tid < 64 ? gb1 : db1)[h * kL + u];
        for (int cc = 0; cc < kD; ++cc) acc = fmaf(bf16_to_f32(w1[kD + cc]), C[cc], acc);
        sC1[tid] = acc;
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

    // c1 values this lane needs: hidden u = 32 mb + 16 (r / 8) + 8 hh + r % 8.
    float c1[4][16];
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) c1[mb][r] = sC1[32 * mb + 16 * (r >> 3) + 8 * hh + (r & 7)];

    for (int64_t tb = t0 + 32 * wave; tb < t1; tb += 128) {
        const int64_t tok = tb + n;
        const bool ok = tok < t1;
        const bf16* vr = V + ((ok ? tok : t0) * H + h) * kD + 8 * hh;
        bf16x8 B[4];
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) B[ks] = load_bf16x8(vr + 16 * ks);
        f32x16 A1[4];
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) {
            A1[mb] = zero_f32x16();
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                const bf16x8 a =
                    *reinterpret_cast<const bf16x8*>(&sW1[(32 * mb + n) * kW + 16 * ks + 8 * hh]);
                A1[mb] = mfma_bf16(a, B[ks], A1[mb]);
            }
        }
        bf16x8 Hop[2][4];   // [gamma|delta][k-step over hidden]
#pragma unroll
        for (int which = 0; which < 2; ++which)
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                const int mb = 2 * which + (ks >> 1), r0 = 8 * (ks & 1);
                float hv[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) hv[j] = act_fn(A1[mb][r0 + j] + c1[mb][r0 + j], act);
                Hop[which][ks] = pack_bf16x8(hv[0], hv[1], hv[2], hv[3], hv[4], hv[5], hv[6], hv[7]);
            }
        f32x16 G[2], D[2];
#pragma unroll
        for (int db = 0; db < 2; ++db) {
            G[db] = zero_f32x16();
            D[db] = zero_f32x16();
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                const bf16x8 ag = *reinterpret_cast<const bf16x8*>(
                    &sW2[0][(32 * db + n) * kW + 16 * ks + 8 * hh]);
                const bf16x8 ad = *reinterpret_cast<const bf16x8*>(
                    &sW2[1][(32 * db + n) * kW + 16 * ks + 8 * hh]);
                G[db] = mfma_bf16(ag, Hop[0][ks], G[db]);
                D[db] = mfma_bf16(ad, Hop[1][ks], D[db]);
            }
        }
        if (ok) {
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
                    if (add_v) {   // identity added: y = v + Eq.7
                        const bf16x4 v = *reinterpret_cast<const bf16x4*>(V + off);
#pragma unroll
                        for (int i = 0; i < 4; ++i) y[i] += (float)v[i];
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
    }
}

// ------------------------------------------------------------------------
// K7 (fp32): one token per thread, weights in LDS, plain FMAs in fp32.
// ------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_surrogate_f32(
    const float* __restrict__ V, const uint8_t* __restrict__ modes, const float* __restrict__ ctx,
    const float* __restrict__ gw1, const float* __restrict__ gb1, const float* __restrict__ gw2,
    const float* __restrict__ gb2, const float* __restrict__ dw1, const float* __restrict__ db1,
    const float* __restrict__ dw2, const float* __restrict__ db2, int act, int add_v, int64_t N,
    int H, void* __restrict__ Y, int ydt) {
    const int h = blockIdx.y;
    if (modes[h] != MODE_SURR) return;
    const int64_t t0 = (int64_t)blockIdx.x * kSurrRows;
    const int64_t t1 = (t0 + kSurrRows < N) ? t0 + kSurrRows : N;
    const int tid = threadIdx.x;
    __shared__ float sW1v[2][kL][kD + 1];   // value half of layer 1, [gamma|delta][u][c]
    __shared__ float sW2t[2][kL][kD];       // layer 2 transposed: [which][u][d]
    __shared__ float sC1[2][kL], sC[kD], sB2[2][kD];
    const float* C = ctx + h * kD;
    for (int i = tid; i < 2 * kL * kD; i += 256) {
        const int which = i / (kL * kD), u = (i / kD) % kL, cc = i % kD;
        const float* w1 = (which == 0 ? gw1 : dw1) + ((int64_t)h * kL + u) * 2 * kD;
        sW1v[which][u][cc] = w1[cc];
        const float* w2 = (which == 0 ? gw2 : dw2) + (int64_t)h * kD * kL;
        // sW2t[which][u][d] = W2[d][u]; here (u, cc) runs over (hidden, d)
        sW2t[which][u][cc] = w2[(int64_t)cc * kL + u];
    }
    if (tid < 128) {
        const int which = tid >> 6, u = tid & 63;
        const float* w1 = (which == 0 ? gw1 : dw1) + ((int64_t)h * kL + u) * 2 * kD;
        float acc = (which == 0 ? gb1 : db1)[h * kL + u];
        for (int cc = 0; cc < kD; ++cc) acc = fmaf(w1[kD + cc], C[cc], acc);
        sC1[which][u] = acc;
    }
    if (tid < kD) {
        sC[tid] = C[tid];
        sB2[0][tid] = gb2[h * kD + tid];
        sB2[1][tid] = db2[h * kD + tid];
    }
    __syncthreads();
    for (int64_t tok = t0 + tid; tok < t1; tok += 256) {
        float v[kD], og[kD], od[kD];
        const float* vr = V + (tok * H + h) * kD;
#pragma unroll
        for (int k = 0; k < kD; ++k) {
            v[k] = vr[k];
            og[k] = sB2[0][k];
            od[k] = sB2[1][k];
        }
        for (int u = 0; u < kL; ++u) {
            float ag = sC1[0][u], ad = sC1[1][u];
#pragma unroll
            for (int k = 0; k < kD; ++k) {
                ag = fmaf(sW1v[0][u][k], v[k], ag);
                ad = fmaf(sW1v[1][u][k], v[k], ad);
            }
            const float hg = act_fn(ag, act), hd = act_fn(ad, act);
#pragma unroll
            for (int k = 0; k < kD; ++k) {
                og[k] = fmaf(sW2t[0][u][k], hg, og[k]);
                od[k] = fmaf(sW2t[1][u][k], hd, od[k]);
            }
        }
        const int64_t off = (tok * H + h) * kD;
#pragma unroll
        for (int k = 0; k < kD; ++k) {
            const float y = sC[k] + sigmoid_fast(og[k]) * od[k] + (add_v ? v[k] : 0.f);
            if (ydt == DT_BF16)
                reinterpret_cast<bf16*>(Y)[off + k] = (bf16)y;
            else
                reinterpret_cast<float*>(Y)[off + k] = y;
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
// Three kernels, fp32 arithmetic throughout (HBM-bound: each of Q, K, V is
// read once):
//   K10a  per (token chunk, head): partial S and z of the chunk;
//   K10b  per head: S and z summed over the chunks in chunk order;
//   K10c  per (token block, head): y_i, one token per thread, S in LDS.
// ------------------------------------------------------------------------
__device__ __forceinline__ float elu1(float x) {
    return x > 0.f ? x + 1.f : exp2f_fast(x * kLog2e);
}

// 16 consecutive values of row `row` of a [N, H, 64] tensor, as fp32.
template <int DT>
__device__ __forceinline__ void load16(const void* __restrict__ X, int64_t off, float* o) {
    if (DT == DT_BF16) {
        const bf16* p = reinterpret_cast<const bf16*>(X) + off;
        const bf16x8 a = load_bf16x8(p), b = load_bf16x8(p + 8);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            o[j] = bf16_to_f32(a[j]);
            o[8 + j] = bf16_to_f32(b[j]);
        }
    } else {
        const float4* p = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(X) + off);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float4 v = p[j];
            o[4 * j] = v.x; o[4 * j + 1] = v.y; o[4 * j + 2] = v.z; o[4 * j + 3] = v.w;
        }
    }
}

// K10a.  Thread t owns row e = t / 4 of S and its columns 16 (t % 4) ... +15;
// 64-token tiles of phi(K) and V are staged in LDS (rows past the chunk are
// zero, so they add nothing).
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
    const int tid = threadIdx.x, e = tid >> 2, c0 = (tid & 3) * 16;
    __shared__ __attribute__((aligned(16))) float sK[64][kD];
    __shared__ __attribute__((aligned(16))) float sV[64][kD];
    float acc[16], z = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = 0.f;
    for (int64_t tb = t0; tb < t1; tb += 64) {
        const int64_t tok = tb + e;   // staging: token row e, values c0 ... c0+15
        float kv[16], vv[16];
        if (tok < t1) {
            load16<DT>(K, (tok * H + h) * kD + c0, kv);
            load16<DT>(V, (tok * H + h) * kD + c0, vv);
#pragma unroll
            for (int i = 0; i < 16; ++i) kv[i] = elu1(kv[i]);
        } else {
#pragma unroll
            for (int i = 0; i < 16; ++i) kv[i] = vv[i] = 0.f;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            *reinterpret_cast<float4*>(&sK[e][c0 + 4 * i]) =
                make_float4(kv[4 * i], kv[4 * i + 1], kv[4 * i + 2], kv[4 * i + 3]);
            *reinterpret_cast<float4*>(&sV[e][c0 + 4 * i]) =
                make_float4(vv[4 * i], vv[4 * i + 1], vv[4 * i + 2], vv[4 * i + 3]);
        }
        __syncthreads();
#pragma unroll 4
        for (int j = 0; j < 64; ++j) {
            const float a = sK[j][e];
            z += a;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float4 v = *reinterpret_cast<const float4*>(&sV[j][c0 + 4 * i]);
                acc[4 * i] = fmaf(a, v.x, acc[4 * i]);
                acc[4 * i + 1] = fmaf(a, v.y, acc[4 * i + 1]);
                acc[4 * i + 2] = fmaf(a, v.z, acc[4 * i + 2]);
                acc[4 * i + 3] = fmaf(a, v.w, acc[4 * i + 3]);
            }
        }
        __syncthreads();
    }
    float* o = part + ((int64_t)h * gridDim.x + c) * kLinSums;
#pragma unroll
    for (int i = 0; i < 4; ++i)
        *reinterpret_cast<float4*>(o + e * kD + c0 + 4 * i) =
            make_float4(acc[4 * i], acc[4 * i + 1], acc[4 * i + 2], acc[4 * i + 3]);
    if ((tid & 3) == 0) o[kD * kD + e] = z;
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

// K10c.  One token per thread: phi(q) in registers, S and z broadcast from
// LDS, 64 x 64 FMAs per token.
template <int DT>
__global__ __launch_bounds__(256) void k_linattn_apply(const void* __restrict__ Q,
                                                       const uint8_t* __restrict__ modes,
                                                       const float* __restrict__ sums, int64_t N,
                                                       int H, void* __restrict__ Y, int ydt) {
    const int h = blockIdx.y;
    if (modes[h] != MODE_SURR) return;
    __shared__ __attribute__((aligned(16))) float sS[kLinSums];
    const float* src = sums + h * kLinSums;
    for (int i = threadIdx.x; i < kLinSums; i += 256) sS[i] = src[i];
    __syncthreads();
    const int64_t tok = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (tok >= N) return;
    float fq[kD], y[kD];
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) load16<DT>(Q, (tok * H + h) * kD + 16 * s4, fq + 16 * s4);
#pragma unroll
    for (int k = 0; k < kD; ++k) {
        fq[k] = elu1(fq[k]);
        y[k] = 0.f;
    }
    float den = 0.f;
#pragma unroll
    for (int e = 0; e < kD; ++e) {
        const float a = fq[e];
        den = fmaf(a, sS[kD * kD + e], den);
#pragma unroll
        for (int k = 0; k < kD; k += 4) {
            const float4 s = *reinterpret_cast<const float4*>(&sS[e * kD + k]);
            y[k] = fmaf(a, s.x, y[k]);
            y[k + 1] = fmaf(a, s.y, y[k + 1]);
            y[k + 2] = fmaf(a, s.z, y[k + 2]);
            y[k + 3] = fmaf(a, s.w, y[k + 3]);
        }
    }
    const float inv = 1.f / den;
    const int64_t off = (tok * H + h) * kD;
    if (ydt == DT_BF16) {
#pragma unroll
        for (int k = 0; k < kD; k += 8)
            *reinterpret_cast<bf16x8*>(reinterpret_cast<bf16*>(Y) + off + k) =
                pack_bf16x8(y[k] * inv, y[k + 1] * inv, y[k + 2] * inv, y[k + 3] * inv,
                            y[k + 4] * inv, y[k + 5] * inv, y[k + 6] * inv, y[k + 7] * inv);
    } else {
#pragma unroll
        for (int k = 0; k < kD; k += 4)
            *reinterpret_cast<float4*>(reinterpret_cast<float*>(Y) + off + k) =
                make_float4(y[k] * inv, y[k + 1] * inv, y[k + 2] * inv, y[k + 3] * inv);
    }
}

// ------------------------------------------------------------------ launchers

void launch_linear_heads(const AttnArgs& a, hipStream_t st) {
    const unsigned nbs = (unsigned)((a.N + kSurrRows - 1) / kSurrRows);
    const int v = a.variant;
    if (v == SURR_EQ7 || v == SURR_MEAN_CONTEXT || v == SURR_ADD_IDENTITY) {
        const float* C = v == SURR_MEAN_CONTEXT ? a.vmean : a.ctx;
        const int add_v = v == SURR_ADD_IDENTITY;
        if (a.dtype == DT_BF16)
            hipLaunchKernelGGL(k_surrogate_bf16, dim3(nbs, a.H), dim3(256), 0, st,
                               (const bf16*)a.V, a.modes, C, (const bf16*)a.g_w1, a.g_b1,
                               (const bf16*)a.g_w2, a.g_b2, (const bf16*)a.d_w1, a.d_b1,
                               (const bf16*)a.d_w2, a.d_b2, a.act, add_v, a.N, a.H, a.Y, a.ydt);
        else
            hipLaunchKernelGGL(k_surrogate_f32, dim3(nbs, a.H), dim3(256), 0, st,
                               (const float*)a.V, a.modes, C, (const float*)a.g_w1, a.g_b1,
                               (const float*)a.g_w2, a.g_b2, (const float*)a.d_w1, a.d_b1,
                               (const float*)a.d_w2, a.d_b2, a.act, add_v, a.N, a.H, a.Y, a.ydt);
    } else if (v == SURR_NO_RESIDUAL) {
        const unsigned nb = (unsigned)((a.N + kMeanRows - 1) / kMeanRows);
        hipLaunchKernelGGL(k_broadcast_heads, dim3(nb, a.H), dim3(256), 0, st, a.modes,
                           (int)MODE_SURR, a.ctx, a.N, a.H, a.Y, a.ydt);
    } else {   // SURR_LINEAR_ATTN
        const dim3 gp((unsigned)a.n3, a.H), gc((kLinSums + 255) / 256, a.H),
            ga((unsigned)((a.N + 255) / 256), a.H);
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
