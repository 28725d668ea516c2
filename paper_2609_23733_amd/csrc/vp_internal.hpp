// Host-side launcher interface between the C ABI (vp_api.hip) and the kernel
// files.  Everything here is internal to libvggtprime.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vp {

struct RouterArgs {
    int dtype;
    const void *Q, *K, *V, *W, *U, *w;
    int64_t N;
    int H;
    int64_t n1, chunk1;   // pooling chunks
    float* part1;
    int64_t n2, chunk2;   // routing chunks
    float* part2;
    float scale;
    int mean_pool;        // 1: q_pool = mean of the queries (W, U, w unused)
    float *q_pool, *stats, *score, *ctx, *vmean;
};

struct AttnArgs {
    int dtype, ydt;
    const void *Q, *K, *V;
    const uint8_t* modes;
    const int32_t* buckets;
    int64_t N;
    int H;
    void* vt;      // packed V^T tiles of FULL heads, fp16, scaled (bf16 only)
    float* vpart;  // per (FULL slot, group of key tiles): max |v| (bf16 only)
    float* vsc;    // per FULL slot: (2^-e, 2^e), the scale of its packed V (bf16 only)
    void* kh;      // packed K tiles of FULL heads, fp16 (bf16 only)
    float* kmax;   // per (FULL slot, 64-key tile): max key norm (bf16 only)
    int32_t* qflag;  // per FULL-head work item: needs the running reference point (bf16 only)
    float* part;     // stream-K partial results of the FULL-head kernel (bf16 only)
    void* Y;
    const float *ctx, *vmean;
    const void *g_w1, *g_w2, *d_w1, *d_w2;
    const float *g_b1, *g_b2, *d_b1, *d_b2;
    int act;
    int variant;          // how SURR heads are computed (vp_surr_variant)
    int64_t n3, chunk3;   // linear-attention token chunks
    float* lpart;         // linear-attention partial sums [H][n3][kLinSums]
    float* lsum;          // linear-attention sums [H][kLinSums]
    float* off;           // null, or [H, N]: per query o = log2 sum_k 2^x_qk (x the logit
                          // in log2 units), written by the FULL-head kernels (bf16 only)
};

// Per head: the 64 x 64 sum of phi(k) v^T followed by the 64 sums of phi(k).
constexpr int kLinSums = 64 * 64 + 64;
// Surrogate variants (values of vp_surr_variant).
enum { SURR_EQ7 = 0, SURR_MEAN_CONTEXT = 1, SURR_NO_RESIDUAL = 2, SURR_ADD_IDENTITY = 3,
       SURR_LINEAR_ATTN = 4 };

// The dense block around the routed layer (bf16, D = 1024).
struct BlockArgs {
    int64_t T;                       // tokens
    const __bf16 *X, *Y;             // block input; routed-attention output (Y: block_out)
    const int32_t* pos;              // [T, 2] (row, column)
    const float *ln1_w, *ln1_b, *ln2_w, *ln2_b, *ls1, *ls2;
    const __bf16 *w_qkv, *w_o, *w_fc1, *w_fc2;
    const float *b_qkv, *b_o, *b_fc1, *b_fc2;
    float eps, rope_base;
    __bf16 *Q, *K, *V;               // block_qkv outputs [T, D]
    __bf16* Xout;                    // block_out output [T, D]
    __bf16 *ln, *xa, *hid;           // workspace: LN output [T, D], attention update [T, D], FFN hidden [T, 4D]
};

void launch_block_qkv(const BlockArgs& a, hipStream_t st);
void launch_block_out(const BlockArgs& a, hipStream_t st);
// Distillation targets and losses (bf16 layers).
struct TeacherArgs {
    AttnArgs attn;        // every head FULL; Y = fp32 workspace, buckets and attn.off
                          // ([H, N] per-query softmax offsets) in the workspace
    float* colmax;        // [H, N]
    float* smax;          // [H]
    void* delta;          // [N, H, d]
    int delta_dt;
};
struct LossArgs {
    int dtype;
    const void *A, *B;    // router loss: A = K; latent loss: A = D_hat, B = D^T
    const float *q_pool, *stats, *colmax, *smax;
    float scale, lambda;
    int64_t N;
    int H;
    float* part;          // partial sums (distill_part_bytes)
    float* loss;          // [H]
};
void launch_teacher_targets(const TeacherArgs& a, hipStream_t st);
void launch_router_loss(const LossArgs& a, hipStream_t st);
void launch_latent_loss(const LossArgs& a, hipStream_t st);
size_t distill_part_bytes(int H);

// Token merging before the routed attention: the destination / source
// lattice of the bipartite matching, in closed form.  Destinations: every
// token of view 0, the nsp special tokens of every view, and in views 1..
// the patches k (index among the view's np patches) with k % g == 0;
// sources: the other patches.  Destination slots and source indices both
// follow token order.
struct TomeGeom {
    int64_t N, P;     // tokens, tokens per view
    int64_t nsp, np;  // special tokens and patches per view
    int64_t g;        // patch stride of the destinations
    int64_t ndp;      // destination patches per view (views 1..)
    int64_t nsv;      // sources per view (views 1..)
    int64_t nD, nA;   // destinations, sources
};
__host__ __device__ inline int64_t tome_dst_token(const TomeGeom& G, int64_t j) {
    if (j < G.P) return j;
    const int64_t per = G.nsp + G.ndp, jj = j - G.P, q = jj / per, w = jj - q * per;
    return (1 + q) * G.P + (w < G.nsp ? w : G.nsp + (w - G.nsp) * G.g);
}
__host__ __device__ inline int64_t tome_src_token(const TomeGeom& G, int64_t i) {
    const int64_t q = i / G.nsv, w = i - q * G.nsv;
    const int64_t b = w / (G.g - 1), o = w - b * (G.g - 1);
    return (1 + q) * G.P + G.nsp + b * G.g + 1 + o;
}
// Destination slot of token t (>= 0), or -1 - (source index) for a source.
__host__ __device__ inline int64_t tome_slot(const TomeGeom& G, int64_t t) {
    if (t < G.P) return t;
    const int64_t v = t / G.P, j = t - v * G.P, per = G.nsp + G.ndp;
    if (j < G.nsp) return G.P + (v - 1) * per + j;
    const int64_t k = j - G.nsp, q = k / G.g, r = k - q * G.g;
    if (r == 0) return G.P + (v - 1) * per + G.nsp + q;
    return -1 - ((v - 1) * G.nsv + q * (G.g - 1) + r - 1);
}
struct TomeArgs {
    TomeGeom G;
    int64_t M;             // sources to merge (rows = N - M)
    const __bf16* K;       // [N, H, 64]
    int H;
    int32_t* row;          // [N]
    int32_t* row_start;    // [N - M + 1]
    int32_t* members;      // [N]
    int32_t* best;         // [N] or null
    float* score;          // [N] or null
    void* ws;              // tome_workspace_bytes(N)
};
size_t tome_workspace_bytes(int64_t N);
void launch_tome_plan(const TomeArgs& a, hipStream_t st);
void launch_tome_merge(int dt, const void* X, int64_t N, int F, int64_t nrows,
                       const int32_t* row_start, const int32_t* members, void* Xm, hipStream_t st);
void launch_tome_unmerge(int dt, const void* Ym, int64_t nrows, const int32_t* row, int64_t N,
                         int F, void* Y, hipStream_t st);
void launch_tome_merge_qkv(const void* Q, const void* K, const void* V, int64_t N, int F,
                           int64_t nrows, const int32_t* row_start, const int32_t* members,
                           void* Qm, void* Km, void* Vm, hipStream_t st);

void launch_router(const RouterArgs& a, hipStream_t st);
void launch_router_logits(const float* u, const void* Wr, const float* br, int R, int Din,
                          int dtype, float* logits, hipStream_t st);
void launch_assign(const float* scores, int H, int rule, float tl, float th, uint8_t* modes,
                   int32_t* buckets, hipStream_t st);
void launch_gather(const AttnArgs& a, hipStream_t st);
void launch_flash(const AttnArgs& a, hipStream_t st);
void launch_linear_heads(const AttnArgs& a, hipStream_t st);
int flash_q_tile(int dtype);
int flash_stream_groups(int64_t N, int H);
size_t flash_part_bytes(int64_t N, int H);
int flash_f32_splits(int64_t N, int H);
size_t flash_f32_part_bytes(int64_t N, int H);
int64_t flash_vmax_parts(int64_t N);

}  // namespace vp
