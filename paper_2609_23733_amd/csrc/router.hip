// Router of the routed global-attention layer (Section 4.1, Eq.1-3), the
// context/mean reductions that reuse its routing weights (Eq.5; Algorithm 1
// mean branch), the linear-logit mode router of the synthetic workloads and
// the mode assignment (Eq.4).
//
// Every reduction over tokens is split into fixed token chunks whose partial
// results are combined in chunk order by a second kernel: no float atomics,
// so results are bitwise reproducible run to run.
#include <type_traits>

#include "vp_device.hpp"
#include "vp_internal.hpp"

namespace vp {

// tanh(x) * sigmoid(y) = (1 - e^{-2x}) / ((1 + e^{-2x}) (1 + e^{-y})), with x
// clamped to +-15 (tanh is +-1 to fp32 precision there) so that no inf/inf
// arises.  Two exponentials and one reciprocal.
__device__ __forceinline__ float tanh_times_sigmoid(float x, float y) {
    x = fminf(fmaxf(x, -15.f), 15.f);
    float e1 = exp2f_fast(-2.f * kLog2e * x);
    float e2 = exp2f_fast(-kLog2e * y);
    return (1.f - e1) * rcp_fast((1.f + e1) * (1.f + e2));
}

// acc + w tanh(x) sigmoid(y), as w (1 - e1) / ((1 + e1) (1 + e2)): the same
// clamp (a median of three, which also passes NaN through without the
// canonicalising move of fminf/fmaxf) and exponentials as above, the
// numerator and the denominator's product each by one FMA.
__device__ __forceinline__ float add_w_tanh_times_sigmoid(float acc, float w, float x, float y) {
    x = __builtin_amdgcn_fmed3f(x, -15.f, 15.f);
    const float e1 = exp2f_fast(-2.f * kLog2e * x);
    const float e2p1 = exp2f_fast(-kLog2e * y) + 1.f;
    return fmaf(fmaf(-e1, w, w), rcp_fast(fmaf(e1, e2p1, e2p1)), acc);
}

// ------------------------------------------------------------------------
// K1: gated attention pooling, partial sums per (token chunk, head).
// part1[c][h] = (m, l, acc[64]) with m = max_i a_i (log2 units: a * log2 e),
// l = sum_i 2^(a_i - m), acc = sum_i 2^(a_i - m) q_i over the chunk's tokens.
// With `mean_pool` (the mean-query ablation, Table 5) every a_i is 0, so the
// same sums give l = token count, acc = sum_i q_i and the combine returns the
// plain mean of the queries; W, U and w are then not read.
// ------------------------------------------------------------------------

// bf16: per head, [W_h; U_h] (128 x 64) times Q_h^T (64 x 32 tokens) on MFMA.
// The four 32-row blocks of A are W rows 0-31, W rows 32-63, U rows 0-31,
// U rows 32-63, so W and U results for one hidden unit l land in the same
// lane and register.
__global__ __launch_bounds__(256, 3) void k_pool_partial_bf16(const bf16* __restrict__ Q,
                                                           const bf16* __restrict__ W,
                                                           const bf16* __restrict__ U,
                                                           const bf16* __restrict__ w,
                                                           int64_t N, int H, int64_t chunk,
                                                           int mean_pool,
                                                           float* __restrict__ part) {
    const int h = blockIdx.y, c = blockIdx.x;
    const int64_t t0 = (int64_t)c * chunk;
    const int64_t t1 = (t0 + chunk < N) ? t0 + chunk : N;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int n = lane & 31, hh = lane >> 5;

    // W_h rows 0-63 then U_h rows 0-63 (bf16, 144-byte rows) and w_h, staged
    // in LDS for the token loop; the same memory holds the wave partials
    // afterwards.
    __shared__ __attribute__((aligned(16))) float smem[4 * 64 * 33];
    __shared__ float s_ml[4][2];
    bf16* sWU = reinterpret_cast<bf16*>(smem);
    float* sw = smem + 128 * 36;   // after the 128 rows of 72 bf16
    if (!mean_pool) {
        const bf16* Wh = W + (int64_t)h * kL * kD;
        const bf16* Uh = U + (int64_t)h * kL * kD;
        for (int i = threadIdx.x; i < 128 * 8; i += 256) {
            const int row = i >> 3, seg = (i & 7) * 8;
            const bf16* src = (row < 64 ? Wh : Uh) + (row & 63) * kD + seg;
            *reinterpret_cast<bf16x8*>(&sWU[row * 72 + seg]) = load_bf16x8(src);
        }
        if (threadIdx.x < kL) sw[threadIdx.x] = bf16_to_f32(w[(int64_t)h * kL + threadIdx.x]);
    }
    __syncthreads();

    float m = -INFINITY, l = 0.f;
    float acc[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) acc[i] = 0.f;

    // Each wave takes 32 tokens at a time; the next block's Q is loaded while
    // this one is computed.  Tail lanes read a valid row (the chunk's first)
    // and zero it afterwards.
    auto load_q = [&](int64_t tb, bf16x8 (&B)[4]) {
        const int64_t tok = tb + n;
        const bf16* qrow = Q + ((tok < t1 ? tok : t0) * H + h) * kD;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) B[ks] = load_bf16x8(qrow + 16 * ks + 8 * hh);
    };
    // One 32-token block: B holds its tokens' rows (tail lanes hold the
    // chunk's first row, a finite value that p = 0 removes from the sums).
    auto block = [&](int64_t tb, const bf16x8 (&B)[4], auto fixed_tag) {
        const int64_t tok = tb + n;
        const bool valid = tok < t1;
        float a = 0.f;
        if (!mean_pool) {
            // An opaque offset keeps the fragment reads in the loop (hoisted,
            // they would hold 96 registers for the whole loop).
            int frow = n * 72 + 8 * hh;
            asm volatile("" : "+v"(frow));
            f32x16 aW[2], aU[2];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) {
                aW[mb] = zero_f32x16();
                aU[mb] = zero_f32x16();
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    const bf16x8 wop = *reinterpret_cast<const bf16x8*>(
                        &sWU[32 * mb * 72 + frow + 16 * ks]);
                    const bf16x8 uop = *reinterpret_cast<const bf16x8*>(
                        &sWU[(64 + 32 * mb) * 72 + frow + 16 * ks]);
                    aW[mb] = mfma_bf16(wop, B[ks], aW[mb]);
                    aU[mb] = mfma_bf16(uop, B[ks], aU[mb]);
                }
            }
            float pa = 0.f;
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    // hidden units 32 mb + 8 g + 4 hh + i in registers 4 g + i
                    const f32x4 wq = *reinterpret_cast<const f32x4*>(&sw[32 * mb + 8 * g + 4 * hh]);
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        pa = add_w_tanh_times_sigmoid(pa, wq[i], aW[mb][4 * g + i],
                                                      aU[mb][4 * g + i]);
                }
            a = (pa + __shfl_xor(pa, 32)) * kLog2e;
        }
        if (decltype(fixed_tag)::value) {
            // Reference point 0: p = 2^a, |a| <= ||w_h||_1 log2 e.
            const float p = valid ? exp2f_fast(a) : 0.f;
            l += hh == 0 ? p : 0.f;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    acc[8 * ks + j] = fmaf(p, bf16_to_f32(B[ks][j]), acc[8 * ks + j]);
            return;
        }
        if (!valid) a = -INFINITY;
        float bm = a;
#pragma unroll
        for (int o = 16; o >= 1; o >>= 1) bm = fmaxf(bm, __shfl_xor(bm, o));
        const float mn = fmaxf(m, bm);
        const float p = valid ? exp2f_fast(a - mn) : 0.f;
        // (m and mn are the same in every lane: the rescale is skipped, as
        // a whole wave, whenever the block leaves the maximum unchanged.)
        if (__builtin_amdgcn_readfirstlane(mn != m ? 1 : 0)) {
            const float al = exp2f_fast(m - mn);
            l = l * al + (hh == 0 ? p : 0.f);
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    acc[8 * ks + j] = acc[8 * ks + j] * al + p * bf16_to_f32(B[ks][j]);
        } else {
            l += hh == 0 ? p : 0.f;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    acc[8 * ks + j] = fmaf(p, bf16_to_f32(B[ks][j]), acc[8 * ks + j]);
        }
        m = mn;
    };
    auto loop = [&](auto fixed_tag) {
        bf16x8 Bc[4], Bn[4];
        load_q(t0 + 32 * wave, Bc);
        for (int64_t tb = t0 + 32 * wave; tb < t1; tb += 128) {
            load_q(tb + 128 < t1 ? tb + 128 : tb, Bn);
            block(tb, Bc, fixed_tag);
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) Bc[ks] = Bn[ks];
        }
    };
    // While ||w_h||_1 log2 e <= 60 every 2^a lies in [2^-60, 2^60], and the
    // sums need no reference point (m = 0); otherwise a running maximum.
    float wl1 = 0.f;
    if (!mean_pool) {
        wl1 = wave_sum(lane < kL ? fabsf(sw[lane]) : 0.f) * kLog2e;
        wl1 = __builtin_amdgcn_readfirstlane(wl1);
    }
    if (mean_pool || wl1 <= 60.f) {
        m = 0.f;
        loop(std::true_type{});
    } else {
        loop(std::false_type{});
    }
    __syncthreads();   // the staged weights are no longer read

    // Combine lanes (same hh share a d set) and waves through LDS.
    float (*s_acc)[64][33] = reinterpret_cast<float (*)[64][33]>(smem);

    const float lw = wave_sum(l);
#pragma unroll
    for (int i = 0; i < 32; ++i) s_acc[wave][lane][i] = acc[i];
    if (lane == 0) {
        s_ml[wave][0] = m;
        s_ml[wave][1] = lw;
    }
    __syncthreads();
    if (threadIdx.x < 64) {
        const int d = threadIdx.x;
        const int ks = d >> 4, dh = (d >> 3) & 1, j = d & 7;
        float M = -INFINITY;
        for (int wv2 = 0; wv2 < 4; ++wv2) M = fmaxf(M, s_ml[wv2][0]);
        float L = 0.f, A = 0.f;
        for (int wv2 = 0; wv2 < 4; ++wv2) {
            const float mw = s_ml[wv2][0];
            const float sc = (mw == -INFINITY) ? 0.f : exp2f_fast(mw - M);
            L += s_ml[wv2][1] * sc;
            float sa = 0.f;
            for (int nn = 0; nn < 32; ++nn) sa += s_acc[wv2][32 * dh + nn][8 * ks + j];
            A += sa * sc;
        }
        float* o = part + ((int64_t)h * gridDim.x + c) * (2 + kD);
        if (d == 0) {
            o[0] = M;
            o[1] = L;
        }
        o[2 + d] = A;
    }
}

// fp32: the same structure on fp32 32x32x2 MFMAs.  Step s of a 32-token block
// reduces over query features s (lanes hh = 0) and 32 + s (hh = 1), so a lane
// holds one contiguous half of its token's query row (the B operand, and the
// values the pooled sum weights); W and U sit in LDS row-major with stride 65
// floats (the A-operand reads are bank-conflict free).
constexpr int kPoolS = 65;

__global__ __launch_bounds__(256) void k_pool_partial_f32(const float* __restrict__ Q,
                                                          const float* __restrict__ W,
                                                          const float* __restrict__ U,
                                                          const float* __restrict__ w,
                                                          int64_t N, int H, int64_t chunk,
                                                          int mean_pool,
                                                          float* __restrict__ part) {
    const int h = blockIdx.y, c = blockIdx.x;
    const int64_t t0 = (int64_t)c * chunk;
    const int64_t t1 = (t0 + chunk < N) ? t0 + chunk : N;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int n = lane & 31, hh = lane >> 5;

    // W_h rows then U_h rows (stride 65) and w_h for the token loop; the same
    // memory holds the wave partials afterwards.
    __shared__ float smem[4 * 64 * 33];
    __shared__ float sw[kL], s_ml[4][2];
    float* sWU = smem;
    if (!mean_pool) {
        const float* Wh = W + (int64_t)h * kL * kD;
        const float* Uh = U + (int64_t)h * kL * kD;
        for (int i = threadIdx.x; i < 2 * kL * kD; i += 256) {
            const int row = i / kD, col = i % kD;
            sWU[row * kPoolS + col] = (row < kL ? Wh : Uh)[(row & (kL - 1)) * kD + col];
        }
        if (threadIdx.x < kL) sw[threadIdx.x] = w[(int64_t)h * kL + threadIdx.x];
    }
    __syncthreads();

    float m = -INFINITY, l = 0.f;
    float acc[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) acc[i] = 0.f;
    for (int64_t tb = t0 + 32 * wave; tb < t1; tb += 128) {
        const int64_t tok = tb + n;
        const bool valid = tok < t1;
        float q[32];
        {
            const float4* qr =
                reinterpret_cast<const float4*>(Q + ((valid ? tok : t0) * H + h) * kD + 32 * hh);
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const float4 v = valid ? qr[k] : make_float4(0.f, 0.f, 0.f, 0.f);
                q[4 * k] = v.x; q[4 * k + 1] = v.y; q[4 * k + 2] = v.z; q[4 * k + 3] = v.w;
            }
        }
        float a = 0.f;
        if (!mean_pool) {
            f32x16 aW[2], aU[2];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) aW[mb] = aU[mb] = zero_f32x16();
#pragma unroll
            for (int st = 0; st < 32; ++st)
#pragma unroll
                for (int mb = 0; mb < 2; ++mb) {
                    const int r = (32 * mb + n) * kPoolS + 32 * hh + st;
                    aW[mb] = mfma_f32(sWU[r], q[st], aW[mb]);
                    aU[mb] = mfma_f32(sWU[kL * kPoolS + r], q[st], aU[mb]);
                }
            float pa = 0.f;
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int g = 0; g < 4; ++g)
#pragma unroll
                    for (int i = 0; i < 4; ++i)   // hidden unit 32 mb + 8 g + 4 hh + i
                        pa += sw[32 * mb + 8 * g + 4 * hh + i] *
                              tanh_times_sigmoid(aW[mb][4 * g + i], aU[mb][4 * g + i]);
            a = (pa + __shfl_xor(pa, 32)) * kLog2e;
        }
        if (!valid) a = -INFINITY;
        float bm = a;
#pragma unroll
        for (int o = 16; o >= 1; o >>= 1) bm = fmaxf(bm, __shfl_xor(bm, o));
        const float mn = fmaxf(m, bm);
        const float al = exp2f_fast(m - mn);
        const float p = valid ? exp2f_fast(a - mn) : 0.f;
        l = l * al + (hh == 0 ? p : 0.f);
#pragma unroll
        for (int j = 0; j < 32; ++j) acc[j] = acc[j] * al + p * q[j];
        m = mn;
    }
    __syncthreads();   // the staged weights are no longer read

    // Combine lanes (lanes of one half hold the same 32 features) and waves.
    float (*s_acc)[64][33] = reinterpret_cast<float (*)[64][33]>(smem);
    const float lw = wave_sum(l);
#pragma unroll
    for (int j = 0; j < 32; ++j) s_acc[wave][lane][j] = acc[j];
    if (lane == 0) {
        s_ml[wave][0] = m;
        s_ml[wave][1] = lw;
    }
    __syncthreads();
    if (threadIdx.x < kD) {
        const int d = threadIdx.x, dh = d >> 5, j = d & 31;
        float M = -INFINITY;
        for (int wv = 0; wv < 4; ++wv) M = fmaxf(M, s_ml[wv][0]);
        float L = 0.f, A = 0.f;
        for (int wv = 0; wv < 4; ++wv) {
            const float mw = s_ml[wv][0];
            const float sc = (mw == -INFINITY) ? 0.f : exp2f_fast(mw - M);
            L += s_ml[wv][1] * sc;
            float sa = 0.f;
            for (int nn = 0; nn < 32; ++nn) sa += s_acc[wv][32 * dh + nn][j];
            A += sa * sc;
        }
        float* o = part + ((int64_t)h * gridDim.x + c) * (2 + kD);
        if (d == 0) {
            o[0] = M;
            o[1] = L;
        }
        o[2 + d] = A;
    }
}

// Combine of per-chunk online-softmax partials (m_c, l_c, a_c[...]) of one
// head: M = max_c m_c, w_c = 2^(m_c - M), L = sum_c w_c l_c,
// A = sum_c w_c a_c (and, when `plain` is set, an unweighted sum of a second
// vector).  256 threads: thread (d, g) sums the g-th quarter of the chunks in
// order for feature d; quarters and the L partials are then added in a fixed
// order, so the result does not depend on scheduling.
struct Combined {
    float M, L;
};

// NG groups of 64 threads (the workgroup is 64 NG threads); group g sums a
// contiguous run of chunks, and the groups' sums are added in group order.
template <int NV, int NG>
__device__ Combined combine_chunks(const float* __restrict__ part, int nchunks, int stride,
                                   float (&acc)[NV]) {
    __shared__ float s_w[1024];
    __shared__ float s_red[NG][kD * NV];
    __shared__ float s_ml[2 * NG];
    const int t = threadIdx.x, d = t & 63, g = t >> 6;
    float M = -INFINITY;
    for (int c = t; c < nchunks; c += 64 * NG) M = fmaxf(M, part[(int64_t)c * stride]);
    M = wave_max(M);
    if ((t & 63) == 0) s_ml[g] = M;
    __syncthreads();
    M = s_ml[0];
#pragma unroll
    for (int i = 1; i < NG; ++i) M = fmaxf(M, s_ml[i]);
    for (int c = t; c < nchunks; c += 64 * NG) {
        const float mc = part[(int64_t)c * stride];
        s_w[c] = (mc == -INFINITY) ? 0.f : exp2f_fast(mc - M);
    }
    __syncthreads();
    const int q = (nchunks + NG - 1) / NG;
    const int c0 = g * q, c1 = (c0 + q < nchunks) ? c0 + q : nchunks;
    float a[NV], lsum = 0.f;
#pragma unroll
    for (int v = 0; v < NV; ++v) a[v] = 0.f;
#pragma unroll 4
    for (int c = c0; c < c1; ++c) {
        const float* p = part + (int64_t)c * stride;
        const float w = s_w[c];
        if (d == 0) lsum = fmaf(p[1], w, lsum);
        a[0] = fmaf(p[2 + d], w, a[0]);
        if (NV > 1) a[NV - 1] += p[2 + kD + d];
    }
#pragma unroll
    for (int v = 0; v < NV; ++v) s_red[g][v * kD + d] = a[v];
    if (d == 0) s_ml[NG + g] = lsum;
    __syncthreads();
    Combined r;
    r.M = M;
    r.L = s_ml[NG];
#pragma unroll
    for (int i = 1; i < NG; ++i) r.L += s_ml[NG + i];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
        acc[v] = s_red[0][v * kD + d];
#pragma unroll
        for (int i = 1; i < NG; ++i) acc[v] += s_red[i][v * kD + d];
    }
    return r;
}

// K9a: q_pool_h = (sum_c w_c acc_c) / (sum_c w_c l_c).
__global__ __launch_bounds__(256) void k_pool_combine(const float* __restrict__ part, int nchunks,
                                                      float* __restrict__ q_pool) {
    const int h = blockIdx.x;
    float acc[1];
    const Combined r =
        combine_chunks<1, 4>(part + (int64_t)h * nchunks * (2 + kD), nchunks, 2 + kD, acc);
    if (threadIdx.x < kD) q_pool[h * kD + threadIdx.x] = acc[0] / r.L;
}

// ------------------------------------------------------------------------
// K2: single-query attention of q_pool over all keys, fused with the context
// C_h = r_h V_h and the value sum, partial per token chunk, all heads.
// part2[c][h] = (m, l, C[64], sumv[64]); m in log2 units of t = scale q.k.
// Thread layout: 8 lanes per (token, head) row, each owning 8 of the 64
// values; a workgroup streams whole token rows ([H, 64] contiguous).
// ------------------------------------------------------------------------
constexpr int kRouteThreads = 512;
template <int DT>
__global__ __launch_bounds__(kRouteThreads) void k_route_partial(const void* __restrict__ Kp,
                                                       const void* __restrict__ Vp,
                                                       const float* __restrict__ q_pool,
                                                       float scale, int64_t N, int H,
                                                       int64_t chunk, float* __restrict__ part) {
    const int c = blockIdx.x;
    const int64_t t0 = (int64_t)c * chunk;
    const int64_t t1 = (t0 + chunk < N) ? t0 + chunk : N;
    const int tpr = H * 8;
    const int rpi = kRouteThreads / tpr;
    const int t = threadIdx.x;
    const int rr = t / tpr, hs = t % tpr, h = hs >> 3, seg = hs & 7;
    const bool active = rr < rpi;

    float qp[8];
    const float cs = scale * kLog2e;
#pragma unroll
    for (int j = 0; j < 8; ++j) qp[j] = active ? q_pool[h * kD + seg * 8 + j] * cs : 0.f;
    float m = -INFINITY, l = 0.f, C[8], sv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) C[j] = sv[j] = 0.f;

    if (active) {
        for (int64_t row = t0 + rr; row < t1; row += rpi) {
            float kv[8], vv[8];
            const int64_t off = (row * H + h) * kD + seg * 8;
            if (DT == DT_BF16) {
                bf16x8 k8 = load_bf16x8(reinterpret_cast<const bf16*>(Kp) + off);
                bf16x8 v8 = load_bf16x8(reinterpret_cast<const bf16*>(Vp) + off);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    kv[j] = bf16_to_f32(k8[j]);
                    vv[j] = bf16_to_f32(v8[j]);
                }
            } else {
                const float4* kq = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(Kp) + off);
                const float4* vq = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(Vp) + off);
                float4 a0 = kq[0], a1 = kq[1], b0 = vq[0], b1 = vq[1];
                kv[0] = a0.x; kv[1] = a0.y; kv[2] = a0.z; kv[3] = a0.w;
                kv[4] = a1.x; kv[5] = a1.y; kv[6] = a1.z; kv[7] = a1.w;
                vv[0] = b0.x; vv[1] = b0.y; vv[2] = b0.z; vv[3] = b0.w;
                vv[4] = b1.x; vv[5] = b1.y; vv[6] = b1.z; vv[7] = b1.w;
            }
            float dot = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) dot = fmaf(qp[j], kv[j], dot);
            dot += __shfl_xor(dot, 1);
            dot += __shfl_xor(dot, 2);
            dot += __shfl_xor(dot, 4);
            const float mn = fmaxf(m, dot);
            const float al = exp2f_fast(m - mn);
            const float p = exp2f_fast(dot - mn);
            l = l * al + p;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                C[j] = C[j] * al + p * vv[j];
                sv[j] += vv[j];
            }
            m = mn;
        }
    }
    // Combine the rpi row phases of each (head, segment) in order.
    __shared__ float s_m[kRouteThreads], s_l[kRouteThreads], s_C[kRouteThreads][9],
        s_s[kRouteThreads][9];
    s_m[t] = m;
    s_l[t] = l;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        s_C[t][j] = C[j];
        s_s[t][j] = sv[j];
    }
    __syncthreads();
    if (rr == 0) {
        float M = -INFINITY;
        for (int q = 0; q < rpi; ++q) M = fmaxf(M, s_m[q * tpr + hs]);
        float L = 0.f, CC[8], SS[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) CC[j] = SS[j] = 0.f;
        for (int q = 0; q < rpi; ++q) {
            const int src = q * tpr + hs;
            const float mq = s_m[src];
            const float sc = (mq == -INFINITY) ? 0.f : exp2f_fast(mq - M);
            L += s_l[src] * sc;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                CC[j] += s_C[src][j] * sc;
                SS[j] += s_s[src][j];
            }
        }
        float* o = part + ((int64_t)h * gridDim.x + c) * (2 + 2 * kD);
        if (seg == 0) {
            o[0] = M;
            o[1] = L;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            o[2 + seg * 8 + j] = CC[j];
            o[2 + kD + seg * 8 + j] = SS[j];
        }
    }
}

// K9b: per head, combine the routing partials (up to 512 chunks, 16 groups of
// 64 threads); write stats, score, ctx, vmean.
constexpr int kRouteCombineGroups = 16;
__global__ __launch_bounds__(64 * kRouteCombineGroups) void k_route_combine(const float* __restrict__ part, int nchunks,
                                                       int64_t N, float* __restrict__ stats,
                                                       float* __restrict__ score,
                                                       float* __restrict__ ctx,
                                                       float* __restrict__ vmean) {
    const int h = blockIdx.x, d = threadIdx.x;
    float acc[2];
    const Combined r = combine_chunks<2, kRouteCombineGroups>(
        part + (int64_t)h * nchunks * (2 + 2 * kD), nchunks, 2 + 2 * kD, acc);
    if (d < kD) {
        ctx[h * kD + d] = acc[0] / r.L;
        vmean[h * kD + d] = acc[1] / (float)N;
    }
    if (d == 0) {
        stats[2 * h] = r.M * kLn2;
        stats[2 * h + 1] = r.L;
        score[h] = 1.f / r.L;
    }
}

// ------------------------------------------------------------------------
// K3: linear-logit mode router, one workgroup per output row, fixed-order
// tree reduction.
// ------------------------------------------------------------------------
template <int DT>
__global__ __launch_bounds__(256) void k_router_logits(const float* __restrict__ u,
                                                       const void* __restrict__ Wr,
                                                       const float* __restrict__ br, int Din,
                                                       float* __restrict__ logits) {
    const int r = blockIdx.x, t = threadIdx.x;
    float acc = 0.f;
    for (int c = t; c < Din; c += 256) {
        const float wv = (DT == DT_BF16)
                             ? bf16_to_f32(reinterpret_cast<const bf16*>(Wr)[(int64_t)r * Din + c])
                             : reinterpret_cast<const float*>(Wr)[(int64_t)r * Din + c];
        acc = fmaf(wv, u[c], acc);
    }
    acc = wave_sum(acc);
    __shared__ float s[4];
    if ((t & 63) == 0) s[t >> 6] = acc;
    __syncthreads();
    if (t == 0) logits[r] = ((s[0] + s[1]) + (s[2] + s[3])) + br[r];
}

// ------------------------------------------------------------------------
// K4: mode per head (Eq.4 or first argmax, or their two-branch MEAN/FULL
// forms of the compute-mode ablation, Table 6) and the grouped head lists.
// ------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_assign(const float* __restrict__ scores, int H, int rule,
                                               float tau_low, float tau_high,
                                               uint8_t* __restrict__ modes,
                                               int32_t* __restrict__ buckets) {
    __shared__ int s_mode[kMaxHeads];
    __shared__ int s_nan[kMaxHeads];
    const int h = threadIdx.x;
    if (h < H) {
        int md, bad = 0;
        if (rule == 0 || rule == 2) {   // Eq.4; rule 2: two-branch (no SURR)
            const float s = scores[h];
            bad = isnan(s);
            md = (bad || s >= tau_high) ? MODE_FULL
                                        : ((rule == 2 || s <= tau_low) ? MODE_MEAN : MODE_SURR);
        } else if (rule == 1) {          // first argmax of the three logits
            const float* lg = scores + 3 * h;
            bad = isnan(lg[0]) || isnan(lg[1]) || isnan(lg[2]);
            md = 0;
            if (lg[1] > lg[md]) md = 1;
            if (lg[2] > lg[md]) md = 2;
            if (bad) md = MODE_FULL;
        } else {                         // rule 3: MEAN vs FULL logit, MEAN on a tie
            const float* lg = scores + 3 * h;
            bad = isnan(lg[MODE_MEAN]) || isnan(lg[MODE_FULL]);
            md = (bad || lg[MODE_FULL] > lg[MODE_MEAN]) ? MODE_FULL : MODE_MEAN;
        }
        s_mode[h] = md;
        s_nan[h] = bad;
        modes[h] = (uint8_t)md;
    }
    __syncthreads();
    if (h == 0) {
        int cnt[3] = {0, 0, 0}, flags = 0;
        for (int i = 0; i < H; ++i) {
            cnt[s_mode[i]]++;
            flags |= s_nan[i];
        }
        int pos = 3;
        for (int md = 0; md < 3; ++md)
            for (int i = 0; i < H; ++i)
                if (s_mode[i] == md) buckets[pos++] = i;
        for (; pos < 3 + kMaxHeads; ++pos) buckets[pos] = -1;
        buckets[0] = cnt[0];
        buckets[1] = cnt[1];
        buckets[2] = cnt[2];
        buckets[3 + kMaxHeads] = flags;
    }
}

// ------------------------------------------------------------------ launchers

void launch_router(const RouterArgs& a, hipStream_t st) {
    const dim3 g1((unsigned)a.n1, (unsigned)a.H);
    if (a.dtype == DT_BF16)
        hipLaunchKernelGGL(k_pool_partial_bf16, g1, dim3(256), 0, st, (const bf16*)a.Q,
                           (const bf16*)a.W, (const bf16*)a.U, (const bf16*)a.w, a.N, a.H,
                           a.chunk1, a.mean_pool, a.part1);
    else
        hipLaunchKernelGGL(k_pool_partial_f32, g1, dim3(256), 0, st, (const float*)a.Q,
                           (const float*)a.W, (const float*)a.U, (const float*)a.w, a.N, a.H,
                           a.chunk1, a.mean_pool, a.part1);
    hipLaunchKernelGGL(k_pool_combine, dim3(a.H), dim3(256), 0, st, a.part1, (int)a.n1,
                       a.q_pool);
    if (a.dtype == DT_BF16)
        hipLaunchKernelGGL(k_route_partial<DT_BF16>, dim3((unsigned)a.n2), dim3(kRouteThreads), 0, st, a.K,
                           a.V, a.q_pool, a.scale, a.N, a.H, a.chunk2, a.part2);
    else
        hipLaunchKernelGGL(k_route_partial<DT_F32>, dim3((unsigned)a.n2), dim3(kRouteThreads), 0, st, a.K,
                           a.V, a.q_pool, a.scale, a.N, a.H, a.chunk2, a.part2);
    hipLaunchKernelGGL(k_route_combine, dim3(a.H), dim3(64 * kRouteCombineGroups), 0, st, a.part2, (int)a.n2, a.N,
                       a.stats, a.score, a.ctx, a.vmean);
}

void launch_router_logits(const float* u, const void* Wr, const float* br, int R, int Din,
                          int dtype, float* logits, hipStream_t st) {
    if (dtype == DT_BF16)
        hipLaunchKernelGGL(k_router_logits<DT_BF16>, dim3(R), dim3(256), 0, st, u, Wr, br, Din,
                           logits);
    else
        hipLaunchKernelGGL(k_router_logits<DT_F32>, dim3(R), dim3(256), 0, st, u, Wr, br, Din,
                           logits);
}

void launch_assign(const float* scores, int H, int rule, float tl, float th, uint8_t* modes,
                   int32_t* buckets, hipStream_t st) {
    hipLaunchKernelGGL(k_assign, dim3(1), dim3(64), 0, st, scores, H, rule, tl, th, modes,
                       buckets);
}

}  // namespace vp
