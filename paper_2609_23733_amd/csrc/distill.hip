// Distillation targets and losses (Section 4.4, Eq.8-11), bf16 layers.
//   Eq.8  p^T_{h,k} = max over queries q of A_{h,k,q}, A_h the teacher's
//         post-softmax attention (every query attends all N keys);
//         s^attn_h = max_k p^T_{h,k};
//   Eq.10 Delta^T_h = (A_h - I) V_h;
//   Eq.9  router loss  KL(p_bar || r_bar) + lambda |max p^T - max r|;
//   Eq.11 latent loss  ||D_hat - D^T|| + lambda (1 - cos(D_hat, D^T)).
// The column maxima take two passes over all (query, key) pairs:
//   D1  per query, o_q = log2 sum_k 2^x_qk (x the logit in log2 units), its
//       softmax normaliser: written by the teacher instances of the FULL-head
//       kernels, which compute Delta^T's attention in the same pass;
//   D2  per key, max over queries of x_qk - o_q, exponentiated once at the
//       end (exp2 is monotone, so the maximum can be taken before it), on the
//       bf16 MFMA (bf16 products are exact in fp32).
#include "vp_device.hpp"
#include "vp_internal.hpp"

namespace vp {

constexpr int kDL = 72;   // bf16 LDS row stride (144 B)

// ------------------------------------------------------------------------
// D2: one workgroup = kCmWaves waves x (32 kCmKB) keys of one head; each wave
// keeps its key rows as the MFMA's A operand in registers.  Query tiles of
// 32 kCmQB (Q rows and -o_q / c) are staged through LDS, double-buffered, and
// shared by the waves.  The accumulator starts at -o_q / c, so the MFMA
// returns (x_qk - o_q) / c and a score costs half of a three-way max (two
// query blocks at once); c > 0 carries the maximum over to x - o.  Queries
// past N carry -inf; keys past N read row 0 and are not written.
// ------------------------------------------------------------------------
constexpr int kCmWaves = 8;
constexpr int kCmKB = 2;                            // 32-key blocks per wave
constexpr int kCmQB = 2;                            // 32-query blocks per tile (even)
constexpr int kCmKeys = 32 * kCmKB * kCmWaves;      // keys per workgroup
constexpr int kCmQ = 32 * kCmQB;                    // queries per LDS tile

__global__ __launch_bounds__(64 * kCmWaves) void k_colmax(const bf16* __restrict__ Q,
                                                          const bf16* __restrict__ K,
                                                          const float* __restrict__ off,
                                                          int64_t N, int H, float c,
                                                          float* __restrict__ colmax) {
    constexpr int kThreads = 64 * kCmWaves;
    constexpr int kSegs = kCmQ * 8 / kThreads;   // 16-byte tile segments per thread
    static_assert(kSegs * kThreads == kCmQ * 8 && kCmQ <= kThreads && kCmQB % 2 == 0, "tile");
    const int h = blockIdx.y;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, n = lane & 31, hh = lane >> 5;
    const int64_t k0 = (int64_t)blockIdx.x * kCmKeys + wave * 32 * kCmKB;
    bf16x8 Ka[kCmKB][4];
#pragma unroll
    for (int kb = 0; kb < kCmKB; ++kb) {
        const int64_t key = k0 + 32 * kb + n;
        const bf16* kp = K + ((key < N ? key : 0) * H + h) * kD + 8 * hh;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) Ka[kb][ks] = load_bf16x8(kp + 16 * ks);
    }
    __shared__ __attribute__((aligned(16))) bf16 sQ[2][kCmQ * kDL];
    __shared__ float sO[2][kCmQ];
    const float* oh = off + (int64_t)h * N;
    const float ninv = -1.f / c;
    bf16x8 gq[kSegs];
    float go = 0.f;
    // (Token indices fit int32: N is at most 2^28.)
    const int Ni = (int)N;
    const int64_t qstride = (int64_t)H * kD;
    const bf16* qh = Q + (int64_t)h * kD;
    auto gload = [&](int t) {
#pragma unroll
        for (int i = 0; i < kSegs; ++i) {
            const int sg = threadIdx.x + i * kThreads;
            const int q = min(t * kCmQ + (sg >> 3), Ni - 1);
            gq[i] = load_bf16x8(qh + (int64_t)q * qstride + (sg & 7) * 8);
        }
        // (scaled at the store, so that nothing waits for the load here)
        if (threadIdx.x < kCmQ) go = oh[min(t * kCmQ + (int)threadIdx.x, Ni - 1)];
    };
    auto lstore = [&](int t, int b) {
#pragma unroll
        for (int i = 0; i < kSegs; ++i) {
            const int sg = threadIdx.x + i * kThreads;
            *reinterpret_cast<bf16x8*>(&sQ[b][(sg >> 3) * kDL + (sg & 7) * 8]) = gq[i];
        }
        if (threadIdx.x < kCmQ)
            sO[b][threadIdx.x] = t * kCmQ + (int)threadIdx.x < Ni ? go * ninv : -INFINITY;
    };
    float acc[kCmKB][16];
#pragma unroll
    for (int kb = 0; kb < kCmKB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[kb][r] = -INFINITY;
    const int nt = (Ni + kCmQ - 1) / kCmQ;
    gload(0);
    lstore(0, 0);
    __syncthreads();
    for (int t = 0; t < nt; ++t) {
        const int b = (int)(t & 1);
        if (t + 1 < nt) gload(t + 1);
#pragma unroll
        for (int qp = 0; qp < kCmQB; qp += 2) {
            // lanes: query (qp + u) * 32 + n of the tile, features 16 ks + 8 hh ..
            bf16x8 qv[2][4];
            f32x16 ci[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int row = (qp + u) * 32 + n;
#pragma unroll
                for (int ks = 0; ks < 4; ++ks)
                    qv[u][ks] = *reinterpret_cast<const bf16x8*>(&sQ[b][row * kDL + 16 * ks + 8 * hh]);
                // ci = 16 copies of o: one copy into a register pair, then
                // 64-bit moves (8 instructions instead of 16).
                const float o = sO[b][row];
                const uint32_t ob = __builtin_bit_cast(uint32_t, o);
                const uint64_t pr = ((uint64_t)ob << 32) | ob;
                uint64_t c8[8];
                c8[0] = pr;
#pragma unroll
                for (int r = 1; r < 8; ++r) asm volatile("v_mov_b64 %0, %1" : "=v"(c8[r]) : "v"(pr));
                ci[u] = __builtin_bit_cast(f32x16, c8);
            }
#pragma unroll
            for (int kb = 0; kb < kCmKB; ++kb) {
                f32x16 Sa = mfma_bf16(Ka[kb][0], qv[0][0], ci[0]);
                f32x16 Sb = mfma_bf16(Ka[kb][0], qv[1][0], ci[1]);
#pragma unroll
                for (int ks = 1; ks < 4; ++ks) {
                    Sa = mfma_bf16(Ka[kb][ks], qv[0][ks], Sa);
                    Sb = mfma_bf16(Ka[kb][ks], qv[1][ks], Sb);
                }
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[kb][r] = fmaxf(acc[kb][r], fmaxf(Sa[r], Sb[r]));
            }
        }
        if (t + 1 < nt) lstore(t + 1, b ^ 1);
        __syncthreads();
    }
    // Maximum over the 32 query lanes of each half (same key rows), then
    // 2^(c max).
#pragma unroll
    for (int kb = 0; kb < kCmKB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float v = acc[kb][r];
#pragma unroll
            for (int o = 1; o < 32; o <<= 1) v = fmaxf(v, __shfl_xor(v, o));
            acc[kb][r] = v;
        }
    if (n == 0) {
#pragma unroll
        for (int kb = 0; kb < kCmKB; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t key = k0 + 32 * kb + 8 * (r >> 2) + 4 * hh + (r & 3);
                if (key < N) colmax[(int64_t)h * N + key] = exp2f(c * acc[kb][r]);
            }
    }
}

// s^attn_h = max_k colmax[h][k]; one workgroup per head.
__global__ __launch_bounds__(256) void k_colmax_max(const float* __restrict__ colmax, int64_t N,
                                                    float* __restrict__ smax) {
    const int h = blockIdx.x;
    float m = 0.f;
    for (int64_t k = threadIdx.x; k < N; k += 256) m = fmaxf(m, colmax[(int64_t)h * N + k]);
    m = wave_max(m);
    __shared__ float s[4];
    if ((threadIdx.x & 63) == 0) s[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) smax[h] = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
}

// Bucket array with every head FULL (the teacher): counts (0, 0, H), ids
// 0 .. H-1, no flags.
__global__ void k_all_full(int H, int32_t* __restrict__ buckets) {
    const int i = threadIdx.x;
    if (i < kBucketsLen) {
        int v = 0;
        if (i == 2) v = H;
        else if (i >= 3 && i < 3 + kMaxHeads) v = (i - 3 < H) ? i - 3 : 0;
        buckets[i] = v;
    }
}

// delta = Y - V (Y fp32, V bf16), rounded once to the output type.
__global__ __launch_bounds__(256) void k_sub_v(const float* __restrict__ Y,
                                               const bf16* __restrict__ V, int64_t n,
                                               void* __restrict__ out, int odt) {
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
    if (i >= n) return;
    const float4 a = *reinterpret_cast<const float4*>(Y + i);
    const float4 b = *reinterpret_cast<const float4*>(Y + i + 4);
    const bf16x8 v = load_bf16x8(V + i);
    float d[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
    for (int j = 0; j < 8; ++j) d[j] -= bf16_to_f32(v[j]);
    if (odt == DT_BF16) {
        *reinterpret_cast<bf16x8*>(reinterpret_cast<bf16*>(out) + i) =
            pack_bf16x8(d[0], d[1], d[2], d[3], d[4], d[5], d[6], d[7]);
    } else {
        float* o = reinterpret_cast<float*>(out) + i;
        *reinterpret_cast<float4*>(o) = make_float4(d[0], d[1], d[2], d[3]);
        *reinterpret_cast<float4*>(o + 4) = make_float4(d[4], d[5], d[6], d[7]);
    }
}

// ------------------------------------------------------------------------
// Eq.9 per head, one pass over the keys: with t_k = scale q_pool . k_k,
// log r_k = t_k - m - log l (router stats), p_k the column maxima and
// P = sum p, the loss is sum p log p / P - log P - sum p log r / P
// + lambda |max p - 1/l|.  Partial sums (P, sum p log p, sum p log r) per
// (key chunk, head), then a fixed-order combine.  8 lanes per key.
// ------------------------------------------------------------------------
constexpr int kLossChunks = 128;

__global__ __launch_bounds__(256) void k_router_loss_partial(
    const bf16* __restrict__ K, const float* __restrict__ q_pool, const float* __restrict__ stats,
    float scale, const float* __restrict__ colmax, int64_t N, int H, float* __restrict__ part) {
    const int h = blockIdx.y, cnk = blockIdx.x;
    const int64_t chunk = (N + kLossChunks - 1) / kLossChunks;
    const int64_t t0 = cnk * chunk, t1 = (t0 + chunk < N) ? t0 + chunk : N;
    const int seg = (threadIdx.x & 7) * 8, rr = threadIdx.x >> 3;
    float qp[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) qp[j] = q_pool[h * kD + seg + j];
    const float m = stats[2 * h], lnl = logf(stats[2 * h + 1]);
    float P = 0.f, Ppp = 0.f, Ppr = 0.f;
    for (int64_t k = t0 + rr; k < t1; k += 32) {
        const bf16x8 kv = load_bf16x8(K + (k * H + h) * kD + seg);
        float dot = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) dot = fmaf(qp[j], bf16_to_f32(kv[j]), dot);
        dot += __shfl_xor(dot, 1);
        dot += __shfl_xor(dot, 2);
        dot += __shfl_xor(dot, 4);
        if ((threadIdx.x & 7) == 0) {
            const float p = colmax[(int64_t)h * N + k];
            const float logr = dot * scale - m - lnl;
            P += p;
            Ppp += p > 0.f ? p * logf(p) : 0.f;
            Ppr += p * logr;
        }
    }
    P = wave_sum(P);
    Ppp = wave_sum(Ppp);
    Ppr = wave_sum(Ppr);
    __shared__ float s[4][3];
    if ((threadIdx.x & 63) == 0) {
        s[threadIdx.x >> 6][0] = P;
        s[threadIdx.x >> 6][1] = Ppp;
        s[threadIdx.x >> 6][2] = Ppr;
    }
    __syncthreads();
    if (threadIdx.x < 3) {
        const int j = threadIdx.x;
        part[((int64_t)h * kLossChunks + cnk) * 3 + j] = (s[0][j] + s[1][j]) + (s[2][j] + s[3][j]);
    }
}

__global__ void k_router_loss_combine(const float* __restrict__ part,
                                      const float* __restrict__ stats,
                                      const float* __restrict__ smax, float lambda, int H,
                                      float* __restrict__ loss) {
    const int h = threadIdx.x;
    if (h >= H) return;
    double P = 0.0, A = 0.0, B = 0.0;
    for (int c = 0; c < kLossChunks; ++c) {
        const float* p = part + ((int64_t)h * kLossChunks + c) * 3;
        P += p[0];
        A += p[1];
        B += p[2];
    }
    const double kl = A / P - log(P) - B / P;
    loss[h] = (float)(kl + (double)lambda * fabs((double)smax[h] - 1.0 / (double)stats[2 * h + 1]));
}

// Eq.11 per head: sums of (a - b)^2, a b, a^2, b^2 over the head's N x d
// entries; partials per (row chunk, head), then a fixed-order combine.
template <int DT>
__global__ __launch_bounds__(256) void k_latent_loss_partial(const void* __restrict__ A,
                                                             const void* __restrict__ B,
                                                             int64_t N, int H,
                                                             float* __restrict__ part) {
    const int h = blockIdx.y, cnk = blockIdx.x;
    const int64_t chunk = (N + kLossChunks - 1) / kLossChunks;
    const int64_t t0 = cnk * chunk, t1 = (t0 + chunk < N) ? t0 + chunk : N;
    const int seg = (threadIdx.x & 7) * 8, rr = threadIdx.x >> 3;
    float sdd = 0.f, sab = 0.f, saa = 0.f, sbb = 0.f;
    for (int64_t t = t0 + rr; t < t1; t += 32) {
        const int64_t o = (t * H + h) * kD + seg;
        float a[8], b[8];
        if (DT == DT_BF16) {
            const bf16x8 x = load_bf16x8(reinterpret_cast<const bf16*>(A) + o);
            const bf16x8 y = load_bf16x8(reinterpret_cast<const bf16*>(B) + o);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                a[j] = bf16_to_f32(x[j]);
                b[j] = bf16_to_f32(y[j]);
            }
        } else {
            const float* x = reinterpret_cast<const float*>(A) + o;
            const float* y = reinterpret_cast<const float*>(B) + o;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                a[j] = x[j];
                b[j] = y[j];
            }
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const float d = a[j] - b[j];
            sdd = fmaf(d, d, sdd);
            sab = fmaf(a[j], b[j], sab);
            saa = fmaf(a[j], a[j], saa);
            sbb = fmaf(b[j], b[j], sbb);
        }
    }
    float v[4] = {wave_sum(sdd), wave_sum(sab), wave_sum(saa), wave_sum(sbb)};
    __shared__ float s[4][4];
    if ((threadIdx.x & 63) == 0)
#pragma unroll
        for (int j = 0; j < 4; ++j) s[threadIdx.x >> 6][j] = v[j];
    __syncthreads();
    if (threadIdx.x < 4) {
        const int j = threadIdx.x;
        part[((int64_t)h * kLossChunks + cnk) * 4 + j] = (s[0][j] + s[1][j]) + (s[2][j] + s[3][j]);
    }
}

__global__ void k_latent_loss_combine(const float* __restrict__ part, float lambda, int H,
                                      float* __restrict__ loss) {
    const int h = threadIdx.x;
    if (h >= H) return;
    double s[4] = {0.0, 0.0, 0.0, 0.0};
    for (int c = 0; c < kLossChunks; ++c)
        for (int j = 0; j < 4; ++j) s[j] += part[((int64_t)h * kLossChunks + c) * 4 + j];
    const double cosv = s[1] / (sqrt(s[2]) * sqrt(s[3]));
    loss[h] = (float)(sqrt(s[0]) + (double)lambda * (1.0 - cosv));
}

// ------------------------------------------------------------------ launchers

size_t distill_part_bytes(int H) { return (size_t)H * kLossChunks * 4 * sizeof(float); }

void launch_teacher_targets(const TeacherArgs& a, hipStream_t st) {
    const float c = kLog2e / sqrtf((float)kD);
    const bf16 *Q = (const bf16*)a.attn.Q, *K = (const bf16*)a.attn.K;
    // D1 with Delta^T's attention: every head FULL into fp32 Y, offsets into
    // attn.off.
    hipLaunchKernelGGL(k_all_full, dim3(1), dim3(64), 0, st, a.attn.H,
                       const_cast<int32_t*>(a.attn.buckets));
    launch_gather(a.attn, st);
    launch_flash(a.attn, st);
    hipLaunchKernelGGL(k_colmax, dim3((unsigned)((a.attn.N + kCmKeys - 1) / kCmKeys), a.attn.H),
                       dim3(64 * kCmWaves), 0, st, Q, K, (const float*)a.attn.off, a.attn.N,
                       a.attn.H, c, a.colmax);
    hipLaunchKernelGGL(k_colmax_max, dim3(a.attn.H), dim3(256), 0, st, (const float*)a.colmax,
                       a.attn.N, a.smax);
    // Delta^T = Y - V.
    const int64_t n = a.attn.N * a.attn.H * kD;
    hipLaunchKernelGGL(k_sub_v, dim3((unsigned)((n / 8 + 255) / 256)), dim3(256), 0, st,
                       (const float*)a.attn.Y, (const bf16*)a.attn.V, n, a.delta, a.delta_dt);
}

void launch_router_loss(const LossArgs& a, hipStream_t st) {
    hipLaunchKernelGGL(k_router_loss_partial, dim3(kLossChunks, a.H), dim3(256), 0, st,
                       (const bf16*)a.A, a.q_pool, a.stats, a.scale, a.colmax, a.N, a.H, a.part);
    hipLaunchKernelGGL(k_router_loss_combine, dim3(1), dim3(64), 0, st, (const float*)a.part,
                       a.stats, a.smax, a.lambda, a.H, a.loss);
}

void launch_latent_loss(const LossArgs& a, hipStream_t st) {
    if (a.dtype == DT_BF16)
        hipLaunchKernelGGL(k_latent_loss_partial<DT_BF16>, dim3(kLossChunks, a.H), dim3(256), 0,
                           st, a.A, a.B, a.N, a.H, a.part);
    else
        hipLaunchKernelGGL(k_latent_loss_partial<DT_F32>, dim3(kLossChunks, a.H), dim3(256), 0,
                           st, a.A, a.B, a.N, a.H, a.part);
    hipLaunchKernelGGL(k_latent_loss_combine, dim3(1), dim3(64), 0, st, (const float*)a.part,
                       a.lambda, a.H, a.loss);
}

}  // namespace vp
