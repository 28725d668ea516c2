// Token merging before the routed attention: ToMe's bipartite soft matching
// (the paper combines its layer with ToMe and gives no steps of its own):
//   T1  metric m_i = bf16(sum over heads of K_{i,h}) (fp32, head order) and
//       1 / |m_i|;
//   T2  for every source, the most similar destination by cosine similarity
//       (MFMA over source x destination tiles, running argmax in registers);
//   T3  the M most similar sources: radix select on unique 64-bit keys
//       (similarity, then the lower token index);
//   T4  rows of the merged sequence (kept tokens in token order), and for
//       each row its tokens: own token first, then its merged sources in
//       token order (stable radix sort of the merged sources by destination);
//   T5  merge = mean of a row's tokens (fp32 sums in member order, one
//       rounding), unmerge = copy of a row's output to each of its tokens.
// Every reduction has a fixed order: results are bitwise reproducible.
#include "vp_device.hpp"
#include "vp_internal.hpp"

namespace vp {

namespace {

constexpr int kRow = 72;           // bf16 LDS row stride (144 B)
constexpr int kScanBlock = 1024;   // elements per scan block (256 threads x 4)
constexpr int kSortBlock = 1024;   // items per radix-sort block (1024 threads x 1)

__device__ __forceinline__ uint64_t lanemask_lt() {
    const int lane = threadIdx.x & 63;
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// Lanes of the wave holding the same 8-bit digit (for an active lane).
__device__ __forceinline__ uint64_t wave_match8(uint32_t d, bool active) {
    uint64_t m = __builtin_amdgcn_ballot_w64(active);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
        const bool bit = (d >> b) & 1u;
        const uint64_t bb = __builtin_amdgcn_ballot_w64(active && bit);
        m &= bit ? bb : ~bb;
    }
    return m;
}

__device__ __forceinline__ uint32_t float_order(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// ---------------------------------------------------------------- T1
// 8 threads per token, 8 features each.
__global__ __launch_bounds__(256) void k_tome_metric(const bf16* __restrict__ K, int64_t N, int H,
                                                     bf16* __restrict__ m,
                                                     float* __restrict__ invn) {
    const int64_t t = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 3;
    const int f = (threadIdx.x & 7) * 8;
    const bool ok = t < N;
    float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (ok)
        for (int h = 0; h < H; ++h) {
            const bf16x8 v = load_bf16x8(K + (t * H + h) * kD + f);
#pragma unroll
            for (int j = 0; j < 8; ++j) s[j] += bf16_to_f32(v[j]);
        }
    bf16x8 o;
    float q = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        o[j] = (bf16)s[j];
        const float x = bf16_to_f32(o[j]);
        q = fmaf(x, x, q);
    }
    q += __shfl_xor(q, 1);
    q += __shfl_xor(q, 2);
    q += __shfl_xor(q, 4);
    if (ok) {
        *reinterpret_cast<bf16x8*>(m + t * kD + f) = o;
        if (f == 0) invn[t] = q > 0.f ? 1.f / sqrtf(q) : 0.f;
    }
}

// ---------------------------------------------------------------- T2
// One workgroup = kTmWaves waves x 64 sources and one chunk of the
// destination tiles (blockIdx.y; chunks split the work finely enough to fill
// the chip); each wave keeps its source rows as the MFMA's A operand.
// Destination tiles of 64 rows (metric, 1 / |m| and a -inf bias past the last
// destination) stream through LDS, double-buffered.  Per score:
// v = dot / |m_d| (an FMA with the bias), a compare and two selects; each
// lane sees its destinations in increasing slot order and keeps the first
// maximum, the final reduction over lanes prefers the lower slot on equal
// values.  The chunk's (value, slot) per source goes to a partial record;
// k_tome_match_final takes the chunks in order (a later chunk wins only when
// strictly larger), so ties still go to the lowest slot.
constexpr int kTmWaves = 4;
constexpr int kTmSrc = 64 * kTmWaves;
constexpr int kTmChunks = 4;          // most destination chunks
constexpr int kTmTargetGroups = 1024; // workgroups the split aims for

__global__ __launch_bounds__(64 * kTmWaves) void k_tome_match(const bf16* __restrict__ m,
                                                              const float* __restrict__ invn,
                                                              TomeGeom G,
                                                              float* __restrict__ pval,
                                                              int32_t* __restrict__ pidx) {
    constexpr int kThreads = 64 * kTmWaves;
    constexpr int kSegs = 64 * 8 / kThreads;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, n = lane & 31, hh = lane >> 5;
    const int64_t i0 = (int64_t)blockIdx.x * kTmSrc + wave * 64;
    bf16x8 A[2][4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
        const int64_t i = i0 + 32 * kb + n;
        const int64_t tok = i < G.nA ? tome_src_token(G, i) : 0;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) A[kb][ks] = load_bf16x8(m + tok * kD + 16 * ks + 8 * hh);
    }
    __shared__ __attribute__((aligned(16))) bf16 sD[2][64 * kRow];
    __shared__ float sInv[2][64], sBias[2][64];
    bf16x8 gq[kSegs];
    float gi = 0.f;
    auto gload = [&](int64_t t) {
#pragma unroll
        for (int s = 0; s < kSegs; ++s) {
            const int sg = threadIdx.x + s * kThreads;
            const int64_t j = t * 64 + (sg >> 3);
            const int64_t tok = j < G.nD ? tome_dst_token(G, j) : 0;
            gq[s] = load_bf16x8(m + tok * kD + (sg & 7) * 8);
        }
        if (threadIdx.x < 64) {
            const int64_t j = t * 64 + threadIdx.x;
            gi = invn[j < G.nD ? tome_dst_token(G, j) : 0];
        }
    };
    auto lstore = [&](int64_t t, int b) {
#pragma unroll
        for (int s = 0; s < kSegs; ++s) {
            const int sg = threadIdx.x + s * kThreads;
            *reinterpret_cast<bf16x8*>(&sD[b][(sg >> 3) * kRow + (sg & 7) * 8]) = gq[s];
        }
        if (threadIdx.x < 64) {
            const bool ok = t * 64 + threadIdx.x < G.nD;
            sInv[b][threadIdx.x] = ok ? gi : 0.f;
            sBias[b][threadIdx.x] = ok ? 0.f : -INFINITY;
        }
    };
    float acc[2][16];
    int32_t idx[2][16];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            acc[kb][r] = -INFINITY;
            idx[kb][r] = 0;
        }
    const int64_t ntt = (G.nD + 63) / 64, C = gridDim.y;
    const int64_t t0 = blockIdx.y * ntt / C, nt = (blockIdx.y + 1) * ntt / C;
    gload(t0);
    lstore(t0, (int)(t0 & 1));
    __syncthreads();
    for (int64_t t = t0; t < nt; ++t) {
        const int b = (int)(t & 1);
        if (t + 1 < nt) gload(t + 1);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            bf16x8 qv[4];
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
                qv[ks] = *reinterpret_cast<const bf16x8*>(
                    &sD[b][(qb * 32 + n) * kRow + 16 * ks + 8 * hh]);
            const float inv = sInv[b][qb * 32 + n], bias = sBias[b][qb * 32 + n];
            const int32_t jn = (int32_t)(t * 64 + qb * 32 + n);
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                f32x16 S = mfma_bf16(A[kb][0], qv[0], zero_f32x16());
#pragma unroll
                for (int ks = 1; ks < 4; ++ks) S = mfma_bf16(A[kb][ks], qv[ks], S);
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const float v = fmaf(S[r], inv, bias);
                    const bool up = v > acc[kb][r];
                    acc[kb][r] = up ? v : acc[kb][r];
                    idx[kb][r] = up ? jn : idx[kb][r];
                }
            }
        }
        if (t + 1 < nt) lstore(t + 1, b ^ 1);
        __syncthreads();
    }
    // Over the 32 destination lanes of each half: the larger value, the
    // lower slot on equal values.
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float v = acc[kb][r];
            int32_t j = idx[kb][r];
#pragma unroll
            for (int o = 1; o < 32; o <<= 1) {
                const float ov = __shfl_xor(v, o);
                const int32_t oj = __shfl_xor(j, o);
                const bool take = ov > v || (ov == v && oj < j);
                v = take ? ov : v;
                j = take ? oj : j;
            }
            acc[kb][r] = v;
            idx[kb][r] = j;
        }
    if (n == 0) {
        const int64_t base = (int64_t)blockIdx.y * G.nA;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t i = i0 + 32 * kb + 8 * (r >> 2) + 4 * hh + (r & 3);
                if (i < G.nA) {
                    pval[base + i] = acc[kb][r];
                    pidx[base + i] = idx[kb][r];
                }
            }
    }
}

// Per source: the best over the chunks, its cosine similarity and its
// selection key (similarity, then the lower token).
__global__ __launch_bounds__(256) void k_tome_match_final(TomeGeom G, int C,
                                                          const float* __restrict__ pval,
                                                          const int32_t* __restrict__ pidx,
                                                          const float* __restrict__ invn,
                                                          int32_t* __restrict__ best,
                                                          float* __restrict__ score,
                                                          uint64_t* __restrict__ key) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= G.nA) return;
    float v = pval[i];
    int32_t j = pidx[i];
    for (int c = 1; c < C; ++c) {
        const float w = pval[(int64_t)c * G.nA + i];
        if (w > v) {
            v = w;
            j = pidx[(int64_t)c * G.nA + i];
        }
    }
    const int64_t tok = tome_src_token(G, i);
    const float sc = v * invn[tok] + 0.f;   // + 0: no -0
    best[i] = j;
    score[i] = sc;
    key[i] = ((uint64_t)float_order(sc) << 32) | (uint64_t)(~(uint32_t)tok);
}

// ---------------------------------------------------------------- T3
// Radix select of the M largest keys, 8 bits per pass from the top.  State:
// [0] prefix (u64), [1] keys still to take (as u64).
__global__ void k_rsel_init(uint64_t* __restrict__ st, uint32_t* __restrict__ ghist, int64_t M) {
    const int i = threadIdx.x;
    if (i < 256) ghist[i] = 0;
    if (i == 0) {
        st[0] = 0;
        st[1] = (uint64_t)M;
    }
}

__global__ __launch_bounds__(256) void k_rsel_hist(const uint64_t* __restrict__ key, int64_t n,
                                                   int shift, const uint64_t* __restrict__ st,
                                                   uint32_t* __restrict__ ghist) {
    __shared__ uint32_t h[256];
    h[threadIdx.x] = 0;
    __syncthreads();
    const uint64_t prefix = st[0];
    const uint64_t hmask = shift >= 56 ? 0ull : (~0ull << (shift + 8));
    const int64_t base = (int64_t)blockIdx.x * 4096;
#pragma unroll 4
    for (int k = 0; k < 16; ++k) {
        const int64_t i = base + k * 256 + threadIdx.x;
        bool act = false;
        uint32_t d = 0;
        if (i < n) {
            const uint64_t v = key[i];
            act = (v & hmask) == (prefix & hmask);
            d = (uint32_t)(v >> shift) & 255u;
        }
        const uint64_t mt = wave_match8(d, act);
        if (act && (mt & lanemask_lt()) == 0) atomicAdd(&h[d], (uint32_t)__popcll(mt));
    }
    __syncthreads();
    if (h[threadIdx.x]) atomicAdd(&ghist[threadIdx.x], h[threadIdx.x]);
}

__global__ void k_rsel_pick(uint64_t* __restrict__ st, uint32_t* __restrict__ ghist, int shift) {
    if (threadIdx.x == 0) {
        const uint64_t rem = st[1];
        uint64_t cum = 0;
        int d = 255;
        for (; d > 0; --d) {
            if (cum + ghist[d] >= rem) break;
            cum += ghist[d];
        }
        st[1] = rem - cum;
        st[0] |= (uint64_t)d << shift;
    }
    __syncthreads();
    if (threadIdx.x < 256) ghist[threadIdx.x] = 0;
}

// ---------------------------------------------------------------- scans
// Exclusive scan of non-negative int32 over n: block sums, a one-workgroup
// scan of the sums, then per-block scans plus their offsets (in == out
// allowed).
__device__ __forceinline__ int block_scan_excl(int v, int* total) {
    __shared__ int ws[4];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == 63) ws[wave] = x;
    __syncthreads();
    int off = 0;
    for (int w = 0; w < wave; ++w) off += ws[w];
    *total = ws[0] + ws[1] + ws[2] + ws[3];
    __syncthreads();
    return off + x - v;
}

__global__ __launch_bounds__(256) void k_scan_sums(const int32_t* __restrict__ in, int64_t n,
                                                   int32_t* __restrict__ bsum) {
    const int64_t i = (int64_t)blockIdx.x * kScanBlock + threadIdx.x * 4;
    int s = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) s += (i + k < n) ? in[i + k] : 0;
    int tot;
    block_scan_excl(s, &tot);
    if (threadIdx.x == 0) bsum[blockIdx.x] = tot;
}

__global__ __launch_bounds__(256) void k_scan_top(int32_t* __restrict__ bsum, int64_t nb,
                                                  int32_t* __restrict__ total) {
    int carry = 0;
    for (int64_t c = 0; c < nb; c += kScanBlock) {
        const int64_t i = c + threadIdx.x * 4;
        int v[4], s = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            v[k] = (i + k < nb) ? bsum[i + k] : 0;
            s += v[k];
        }
        int tot;
        int run = carry + block_scan_excl(s, &tot);
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (i + k < nb) {
                bsum[i + k] = run;
                run += v[k];
            }
        carry += tot;
        __syncthreads();
    }
    if (total && threadIdx.x == 0) *total = carry;
}

__global__ __launch_bounds__(256) void k_scan_apply(const int32_t* in, int64_t n,
                                                    const int32_t* __restrict__ bsum,
                                                    int32_t* out) {
    const int64_t i = (int64_t)blockIdx.x * kScanBlock + threadIdx.x * 4;
    int v[4], s = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        v[k] = (i + k < n) ? in[i + k] : 0;
        s += v[k];
    }
    int tot;
    int run = bsum[blockIdx.x] + block_scan_excl(s, &tot);
#pragma unroll
    for (int k = 0; k < 4; ++k)
        if (i + k < n) {
            out[i + k] = run;
            run += v[k];
        }
}

void scan_excl(const int32_t* in, int32_t* out, int64_t n, int32_t* bsum, int32_t* total,
               hipStream_t st) {
    if (n <= 0) return;
    const int64_t nb = (n + kScanBlock - 1) / kScanBlock;
    hipLaunchKernelGGL(k_scan_sums, dim3((unsigned)nb), dim3(256), 0, st, in, n, bsum);
    hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(256), 0, st, bsum, nb, total);
    hipLaunchKernelGGL(k_scan_apply, dim3((unsigned)nb), dim3(256), 0, st, in, n,
                       (const int32_t*)bsum, out);
}

// ---------------------------------------------------------------- sort
// Stable LSD radix sort of (key, value) pairs by 8-bit digits.
__global__ __launch_bounds__(kSortBlock) void k_rs_hist(const uint32_t* __restrict__ key,
                                                        int64_t n, int shift, int64_t nb,
                                                        int32_t* __restrict__ hist) {
    __shared__ int32_t h[256];
    if (threadIdx.x < 256) h[threadIdx.x] = 0;
    __syncthreads();
    const int64_t i = (int64_t)blockIdx.x * kSortBlock + threadIdx.x;
    const bool act = i < n;
    const uint32_t d = act ? (key[i] >> shift) & 255u : 0u;
    const uint64_t mt = wave_match8(d, act);
    if (act && (mt & lanemask_lt()) == 0) atomicAdd(&h[d], (int32_t)__popcll(mt));
    __syncthreads();
    if (threadIdx.x < 256) hist[(int64_t)threadIdx.x * nb + blockIdx.x] = h[threadIdx.x];
}

__global__ __launch_bounds__(kSortBlock) void k_rs_scatter(const uint32_t* __restrict__ key,
                                                           const int32_t* __restrict__ val,
                                                           int64_t n, int shift, int64_t nb,
                                                           const int32_t* __restrict__ off,
                                                           uint32_t* __restrict__ key_out,
                                                           int32_t* __restrict__ val_out) {
    constexpr int kWaves = kSortBlock / 64;
    __shared__ int32_t wc[kWaves][256];
    for (int k = threadIdx.x; k < kWaves * 256; k += kSortBlock) (&wc[0][0])[k] = 0;
    __syncthreads();
    const int wave = threadIdx.x >> 6;
    const int64_t i = (int64_t)blockIdx.x * kSortBlock + threadIdx.x;
    const bool act = i < n;
    const uint32_t k = act ? key[i] : 0u;
    const uint32_t d = (k >> shift) & 255u;
    const uint64_t mt = wave_match8(d, act);
    const int rank = __popcll(mt & lanemask_lt());
    if (act && rank == 0) wc[wave][d] = __popcll(mt);
    __syncthreads();
    if (act) {
        int64_t pos = off[(int64_t)d * nb + blockIdx.x] + rank;
        for (int w = 0; w < wave; ++w) pos += wc[w][d];
        key_out[pos] = k;
        val_out[pos] = val[i];
    }
}

// ---------------------------------------------------------------- T4
__global__ __launch_bounds__(256) void k_fill_i32(int32_t* __restrict__ p, int64_t n, int32_t v) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) p[i] = v;
}

// Per token: kept flag; per source: merged flag; merged count per
// destination; the optional best / score outputs.
__global__ __launch_bounds__(256) void k_tome_flags(TomeGeom G, const uint64_t* __restrict__ key,
                                                    const uint64_t* __restrict__ st,
                                                    const int32_t* __restrict__ bslot,
                                                    const float* __restrict__ score,
                                                    int32_t* __restrict__ kept,
                                                    int32_t* __restrict__ mflag,
                                                    int32_t* __restrict__ cnt,
                                                    int32_t* __restrict__ best_out,
                                                    float* __restrict__ score_out) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= G.N) return;
    const int64_t s = tome_slot(G, t);
    int k = 1;
    if (s < 0) {
        const int64_t i = -1 - s;
        const int merged = key[i] >= st[0] ? 1 : 0;
        k = 1 - merged;
        mflag[i] = merged;
        if (merged) atomicAdd(&cnt[bslot[i]], 1);
        if (best_out) best_out[t] = (int32_t)tome_dst_token(G, bslot[i]);
        if (score_out) score_out[t] = score[i];
    } else {
        if (best_out) best_out[t] = -1;
        if (score_out) score_out[t] = 0.f;
    }
    kept[t] = k;
}

// Merged sources in token order: (destination slot, token).
__global__ __launch_bounds__(256) void k_tome_compact(TomeGeom G, const int32_t* __restrict__ mflag,
                                                      const int32_t* __restrict__ pos,
                                                      const int32_t* __restrict__ bslot,
                                                      uint32_t* __restrict__ lkey,
                                                      int32_t* __restrict__ lval) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= G.nA || !mflag[i]) return;
    lkey[pos[i]] = (uint32_t)bslot[i];
    lval[pos[i]] = (int32_t)tome_src_token(G, i);
}

// Rows of merged sources (their destination's), and row sizes of kept
// tokens (1 + the sources merged into a destination).
__global__ __launch_bounds__(256) void k_tome_rows(TomeGeom G, const int32_t* __restrict__ kept,
                                                   const int32_t* __restrict__ bslot,
                                                   const int32_t* __restrict__ cnt,
                                                   int32_t* __restrict__ row,
                                                   int32_t* __restrict__ size) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= G.N) return;
    const int64_t s = tome_slot(G, t);
    if (kept[t]) {
        const int64_t r = row[t];
        if (r >= 0 && r < G.N) size[r] = 1 + (s >= 0 ? cnt[s] : 0);
    } else {
        // a kept destination's row is final (it came from the scan)
        row[t] = row[tome_dst_token(G, bslot[-1 - s])];
    }
}

__global__ void k_tome_last(int32_t* __restrict__ row_start, int64_t nrows, int64_t N) {
    if (threadIdx.x == 0) row_start[nrows] = (int32_t)N;
}

// (Every index is checked against its array, so an inconsistent plan cannot
// write outside the caller's buffers.)
__global__ __launch_bounds__(256) void k_tome_members(TomeGeom G, int64_t M, int64_t nrows,
                                                      const int32_t* __restrict__ kept,
                                                      const int32_t* __restrict__ row,
                                                      const int32_t* __restrict__ row_start,
                                                      const uint32_t* __restrict__ skey,
                                                      const int32_t* __restrict__ sval,
                                                      const int32_t* __restrict__ off,
                                                      int32_t* __restrict__ members) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < G.N && kept[i]) {
        const int64_t r = row[i];
        if (r >= 0 && r < nrows) {
            const int64_t p = row_start[r];
            if (p >= 0 && p < G.N) members[p] = (int32_t)i;
        }
    }
    if (i < M) {
        const uint32_t j = skey[i];
        if ((int64_t)j >= G.nD) return;
        const int64_t r = row[tome_dst_token(G, j)];
        if (r < 0 || r >= nrows) return;
        const int64_t p = (int64_t)row_start[r] + 1 + (i - off[j]);
        if (p >= 0 && p < G.N) members[p] = sval[i];
    }
}

// ---------------------------------------------------------------- T5
template <int DT>
__global__ __launch_bounds__(256) void k_tome_merge(const void* __restrict__ X, int64_t N, int F,
                                                    const int32_t* __restrict__ row_start,
                                                    const int32_t* __restrict__ members,
                                                    void* __restrict__ Xm) {
    const int64_t r = blockIdx.x;
    int64_t b = row_start[r], e = row_start[r + 1];
    b = b < 0 ? 0 : (b > N ? N : b);
    e = e < b ? b : (e > N ? N : e);
    for (int f0 = threadIdx.x * 4; f0 < F; f0 += 1024) {
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
        int c = 0;
        for (int64_t p = b; p < e; ++p) {
            const int64_t t = members[p];
            if (t < 0 || t >= N) continue;
            if (DT == DT_BF16) {
                const bf16x4 v = *reinterpret_cast<const bf16x4*>(
                    reinterpret_cast<const bf16*>(X) + t * F + f0);
#pragma unroll
                for (int k = 0; k < 4; ++k) acc[k] += bf16_to_f32(v[k]);
            } else {
                const float4 v = *reinterpret_cast<const float4*>(
                    reinterpret_cast<const float*>(X) + t * F + f0);
                acc[0] += v.x;
                acc[1] += v.y;
                acc[2] += v.z;
                acc[3] += v.w;
            }
            ++c;
        }
        const float cf = c > 0 ? (float)c : 1.f;
        if (DT == DT_BF16) {
            bf16x4 o;
#pragma unroll
            for (int k = 0; k < 4; ++k) o[k] = (bf16)(acc[k] / cf);
            *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(Xm) + r * F + f0) = o;
        } else {
            *reinterpret_cast<float4*>(reinterpret_cast<float*>(Xm) + r * F + f0) =
                make_float4(acc[0] / cf, acc[1] / cf, acc[2] / cf, acc[3] / cf);
        }
    }
}

// Q, K and V of a row at once (bf16, F = 1024 or less): the row's member
// indices are staged in LDS first (256 per pass), so the loads of the three
// tensors do not wait on one index each; sums in member order, as above.
__global__ __launch_bounds__(256) void k_tome_merge_qkv(const bf16* __restrict__ Q,
                                                        const bf16* __restrict__ K,
                                                        const bf16* __restrict__ V, int64_t N,
                                                        int F, const int32_t* __restrict__ row_start,
                                                        const int32_t* __restrict__ members,
                                                        bf16* __restrict__ Qm, bf16* __restrict__ Km,
                                                        bf16* __restrict__ Vm) {
    __shared__ int32_t sm[256];
    const int64_t r = blockIdx.x;
    int64_t b = row_start[r], e = row_start[r + 1];
    b = b < 0 ? 0 : (b > N ? N : b);
    e = e < b ? b : (e > N ? N : e);
    const int f0 = threadIdx.x * 4;
    const bool act = f0 < F;
    float aq[4] = {0.f, 0.f, 0.f, 0.f}, ak[4] = {0.f, 0.f, 0.f, 0.f}, av[4] = {0.f, 0.f, 0.f, 0.f};
    int c = 0;
    for (int64_t p0 = b; p0 < e; p0 += 256) {
        const int cnt = (int)((e - p0) < 256 ? (e - p0) : 256);
        __syncthreads();
        if ((int)threadIdx.x < cnt) sm[threadIdx.x] = members[p0 + threadIdx.x];
        __syncthreads();
        for (int j = 0; j < cnt; ++j) {
            const int64_t t = sm[j];
            if (t < 0 || t >= N) continue;
            ++c;
            if (!act) continue;
            const bf16x4 q = *reinterpret_cast<const bf16x4*>(Q + t * F + f0);
            const bf16x4 k = *reinterpret_cast<const bf16x4*>(K + t * F + f0);
            const bf16x4 v = *reinterpret_cast<const bf16x4*>(V + t * F + f0);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                aq[i] += bf16_to_f32(q[i]);
                ak[i] += bf16_to_f32(k[i]);
                av[i] += bf16_to_f32(v[i]);
            }
        }
    }
    if (!act) return;
    const float cf = c > 0 ? (float)c : 1.f;
    bf16x4 oq, ok, ov;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        oq[i] = (bf16)(aq[i] / cf);
        ok[i] = (bf16)(ak[i] / cf);
        ov[i] = (bf16)(av[i] / cf);
    }
    *reinterpret_cast<bf16x4*>(Qm + r * F + f0) = oq;
    *reinterpret_cast<bf16x4*>(Km + r * F + f0) = ok;
    *reinterpret_cast<bf16x4*>(Vm + r * F + f0) = ov;
}

// 16-byte chunks: Y[t] = Ym[row[t]] (zero for a row outside [0, nrows)).
__global__ __launch_bounds__(256) void k_tome_unmerge(const u32x4* __restrict__ Ym, int64_t nrows,
                                                      const int32_t* __restrict__ row, int64_t N,
                                                      int cpr, u32x4* __restrict__ Y) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= N * cpr) return;
    const int64_t t = i / cpr, c = i - t * cpr;
    const int64_t r = row[t];
    const u32x4 z = {0u, 0u, 0u, 0u};
    Y[i] = (r >= 0 && r < nrows) ? Ym[r * cpr + c] : z;
}

// Workspace of the plan for N tokens.
struct TomeWs {
    size_t m, invn, bslot, score, key, st, ghist, mflag, pos, kept, cnt, off, size, lk0, lv0,
        lk1, lv1, bsum, hist, pval, pidx, total;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

TomeWs tome_ws(int64_t N) {
    TomeWs w;
    const size_t n = (size_t)(N > 0 ? N : 1);
    const size_t nbs = (n + kScanBlock - 1) / kScanBlock + 1;
    const size_t nbr = (n + kSortBlock - 1) / kSortBlock;
    size_t o = 0;
    auto take = [&](size_t bytes) {
        const size_t at = o;
        o = align256(o + bytes);
        return at;
    };
    w.m = take(n * kD * 2);
    w.invn = take(n * 4);
    w.bslot = take(n * 4);
    w.score = take(n * 4);
    w.key = take(n * 8);
    w.st = take(16);
    w.ghist = take(256 * 4);
    w.mflag = take(n * 4);
    w.pos = take(n * 4);
    w.kept = take(n * 4);
    w.cnt = take(n * 4);
    w.off = take(n * 4);
    w.size = take(n * 4);
    w.lk0 = take(n * 4);
    w.lv0 = take(n * 4);
    w.lk1 = take(n * 4);
    w.lv1 = take(n * 4);
    w.bsum = take(((256 * nbr > n ? 256 * nbr : n) / kScanBlock + 2) * 4 + nbs * 4);
    w.hist = take(256 * nbr * 4);
    w.pval = take(n * kTmChunks * 4);
    w.pidx = take(n * kTmChunks * 4);
    w.total = o;
    return w;
}

unsigned grid256(int64_t n) { return (unsigned)((n + 255) / 256); }

}  // namespace

size_t tome_workspace_bytes(int64_t N) { return tome_ws(N).total; }

void launch_tome_plan(const TomeArgs& a, hipStream_t st) {
    const TomeGeom& G = a.G;
    const TomeWs w = tome_ws(G.N);
    char* ws = (char*)a.ws;
    bf16* m = (bf16*)(ws + w.m);
    float* invn = (float*)(ws + w.invn);
    int32_t* bslot = (int32_t*)(ws + w.bslot);
    float* score = (float*)(ws + w.score);
    uint64_t* key = (uint64_t*)(ws + w.key);
    uint64_t* sel = (uint64_t*)(ws + w.st);
    uint32_t* ghist = (uint32_t*)(ws + w.ghist);
    int32_t *mflag = (int32_t*)(ws + w.mflag), *pos = (int32_t*)(ws + w.pos);
    int32_t *kept = (int32_t*)(ws + w.kept), *cnt = (int32_t*)(ws + w.cnt);
    int32_t *off = (int32_t*)(ws + w.off), *size = (int32_t*)(ws + w.size);
    uint32_t *lk0 = (uint32_t*)(ws + w.lk0), *lk1 = (uint32_t*)(ws + w.lk1);
    int32_t *lv0 = (int32_t*)(ws + w.lv0), *lv1 = (int32_t*)(ws + w.lv1);
    int32_t* bsum = (int32_t*)(ws + w.bsum);
    int32_t* hist = (int32_t*)(ws + w.hist);
    const int64_t N = G.N, M = a.M, nrows = N - M;

    hipLaunchKernelGGL(k_rsel_init, dim3(1), dim3(256), 0, st, sel, ghist, M);
    hipLaunchKernelGGL(k_fill_i32, dim3(grid256(G.nD)), dim3(256), 0, st, cnt, G.nD, 0);
    if (G.nA > 0) {
        hipLaunchKernelGGL(k_tome_metric, dim3(grid256(N * 8)), dim3(256), 0, st, a.K, N, a.H, m,
                           invn);
        const int64_t ns = (G.nA + kTmSrc - 1) / kTmSrc, ntt = (G.nD + 63) / 64;
        int64_t C = (kTmTargetGroups + ns - 1) / ns;
        C = C < 1 ? 1 : (C > kTmChunks ? kTmChunks : C);
        C = C > ntt ? ntt : C;
        float* pval = (float*)(ws + w.pval);
        int32_t* pidx = (int32_t*)(ws + w.pidx);
        hipLaunchKernelGGL(k_tome_match, dim3((unsigned)ns, (unsigned)C), dim3(64 * kTmWaves), 0,
                           st, (const bf16*)m, (const float*)invn, G, pval, pidx);
        hipLaunchKernelGGL(k_tome_match_final, dim3(grid256(G.nA)), dim3(256), 0, st, G, (int)C,
                           (const float*)pval, (const int32_t*)pidx, (const float*)invn, bslot,
                           score, key);
        // (M > 0 here: M = 0 leaves stride 1, hence no sources)
        const unsigned gh = (unsigned)((G.nA + 4095) / 4096);
        for (int shift = 56; shift >= 0; shift -= 8) {
            hipLaunchKernelGGL(k_rsel_hist, dim3(gh), dim3(256), 0, st, (const uint64_t*)key, G.nA,
                               shift, (const uint64_t*)sel, ghist);
            hipLaunchKernelGGL(k_rsel_pick, dim3(1), dim3(256), 0, st, sel, ghist, shift);
        }
    }
    hipLaunchKernelGGL(k_tome_flags, dim3(grid256(N)), dim3(256), 0, st, G, (const uint64_t*)key,
                       (const uint64_t*)sel, (const int32_t*)bslot, (const float*)score, kept,
                       mflag, cnt, a.best, a.score);
    // rows of kept tokens
    scan_excl(kept, a.row, N, bsum, nullptr, st);
    if (M > 0) {
        scan_excl(mflag, pos, G.nA, bsum, nullptr, st);
        hipLaunchKernelGGL(k_tome_compact, dim3(grid256(G.nA)), dim3(256), 0, st, G,
                           (const int32_t*)mflag, (const int32_t*)pos, (const int32_t*)bslot, lk0,
                           lv0);
        // stable sort of the merged sources by destination slot
        int bits = 1;
        while (bits < 31 && ((int64_t)1 << bits) < G.nD) ++bits;
        const int64_t nb = (M + kSortBlock - 1) / kSortBlock;
        uint32_t *ki = lk0, *ko = lk1;
        int32_t *vi = lv0, *vo = lv1;
        for (int shift = 0; shift < bits; shift += 8) {
            hipLaunchKernelGGL(k_rs_hist, dim3((unsigned)nb), dim3(kSortBlock), 0, st,
                               (const uint32_t*)ki, M, shift, nb, hist);
            scan_excl(hist, hist, 256 * nb, bsum, nullptr, st);
            hipLaunchKernelGGL(k_rs_scatter, dim3((unsigned)nb), dim3(kSortBlock), 0, st,
                               (const uint32_t*)ki, (const int32_t*)vi, M, shift, nb,
                               (const int32_t*)hist, ko, vo);
            uint32_t* tk = ki;
            ki = ko;
            ko = tk;
            int32_t* tv = vi;
            vi = vo;
            vo = tv;
        }
        lk0 = ki;
        lv0 = vi;
        scan_excl(cnt, off, G.nD, bsum, nullptr, st);
    }
    hipLaunchKernelGGL(k_tome_rows, dim3(grid256(N)), dim3(256), 0, st, G, (const int32_t*)kept,
                       (const int32_t*)bslot, (const int32_t*)cnt, a.row, size);
    scan_excl(size, a.row_start, nrows, bsum, nullptr, st);
    hipLaunchKernelGGL(k_tome_last, dim3(1), dim3(64), 0, st, a.row_start, nrows, N);
    hipLaunchKernelGGL(k_tome_members, dim3(grid256(N)), dim3(256), 0, st, G, M, nrows,
                       (const int32_t*)kept, (const int32_t*)a.row, (const int32_t*)a.row_start,
                       (const uint32_t*)lk0, (const int32_t*)lv0, (const int32_t*)off,
                       a.members);
}

void launch_tome_merge(int dt, const void* X, int64_t N, int F, int64_t nrows,
                       const int32_t* row_start, const int32_t* members, void* Xm,
                       hipStream_t st) {
    if (nrows <= 0) return;
    if (dt == DT_BF16)
        hipLaunchKernelGGL(k_tome_merge<DT_BF16>, dim3((unsigned)nrows), dim3(256), 0, st, X, N, F,
                           row_start, members, Xm);
    else
        hipLaunchKernelGGL(k_tome_merge<DT_F32>, dim3((unsigned)nrows), dim3(256), 0, st, X, N, F,
                           row_start, members, Xm);
}

void launch_tome_merge_qkv(const void* Q, const void* K, const void* V, int64_t N, int F,
                           int64_t nrows, const int32_t* row_start, const int32_t* members,
                           void* Qm, void* Km, void* Vm, hipStream_t st) {
    if (nrows <= 0) return;
    hipLaunchKernelGGL(k_tome_merge_qkv, dim3((unsigned)nrows), dim3(256), 0, st, (const bf16*)Q,
                       (const bf16*)K, (const bf16*)V, N, F, row_start, members, (bf16*)Qm,
                       (bf16*)Km, (bf16*)Vm);
}

void launch_tome_unmerge(int dt, const void* Ym, int64_t nrows, const int32_t* row, int64_t N,
                         int F, void* Y, hipStream_t st) {
    const int cpr = F * (dt == DT_BF16 ? 2 : 4) / 16;
    if (N <= 0) return;
    hipLaunchKernelGGL(k_tome_unmerge, dim3(grid256(N * cpr)), dim3(256), 0, st,
                       (const u32x4*)Ym, nrows, row, N, cpr, (u32x4*)Y);
}

}  // namespace vp
