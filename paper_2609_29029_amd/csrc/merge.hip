// Optional merge of each kept tile's non-selected tokens into contextual tokens
// (Sec. 2.3 Stage 2: VisionZip keeps the dominant tokens and merges the
// remainder; the scheme follows VisionZip).  For kept tile rho with dominant
// tokens sel_idx[sel_offsets[rho] ..) and k_c = ctx_offsets[rho + 1] -
// ctx_offsets[rho] contextual tokens: the remainder R is the other tokens in
// ascending order, target j is R[floor(j |R| / k_c)], every other token of R
// joins the target j of largest cdot(x_r, x_j) * inv_j (ties to the lower j),
// and contextual token j is the float64 sum of its group in ascending index
// order over the group size, rounded to float32 and then to the storage type.
// cdot is the float64 dot product in 8-element granules, granule g into
// accumulator g mod 4, ascending, then (a0 + a2) + (a1 + a3); inv_j is
// 1/sqrt(cdot(x_j, x_j)), 0 for an all-zero token.
//
//   merge_prep    one workgroup per kept tile: the remainder and the targets
//                 (LDS), each token's role in grp (-1 dominant, j for target j,
//                 -2 to be assigned), the targets' inv (lanes r + 16 q: token
//                 r's granule class q, the layout of the score pass).
//                 Workgroup 0 also checks the offsets, tile ids and counts of
//                 the whole call and writes the status word; a tile that fails
//                 its own checks (those, or a dominant index out of range or
//                 repeated) is marked not ok and skipped by the next kernels.
//   merge_assign  grid (64-token chunk of the remainder, tile): 64 tokens per
//                 workgroup, four lanes each (granule classes), every target in
//                 blocks of 32 staged through LDS in 512-element slices; float64
//                 accumulators stay in registers across slices; then the fold,
//                 the score and a running arg-max; writes grp of the token.
//   merge_mean    one workgroup per contextual row: its tile and j by binary
//                 search over ctx_offsets, the group's members (ascending) from
//                 grp, float64 sums of 8-element slices per thread.  Its
//                 workgroup 0 also sets the status word to RIFT_ERR_SHAPE when
//                 merge_prep marked a tile not ok (it runs after merge_prep, so
//                 the two plain stores are ordered).
#include "launch.h"
#include "rift_common.h"

namespace rift {

namespace {

constexpr int kTB = 32;     // targets per LDS block
constexpr int kDC = 512;    // elements per LDS slice

// 8 consecutive stored elements widened to float64 (bf16 or f32)
template <bool BF16>
__device__ __forceinline__ void load8(const void* base, size_t elem, double (&v)[8]) {
    if constexpr (BF16) {
        const u32x4_t w = *reinterpret_cast<const u32x4_t*>(static_cast<const bf16_t*>(base) + elem);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = (double)bf16_lo(w[i]);
            v[2 * i + 1] = (double)bf16_hi(w[i]);
        }
    } else {
        const float* p = static_cast<const float*>(base) + elem;
        const f32x4_t a = *reinterpret_cast<const f32x4_t*>(p);
        const f32x4_t b = *reinterpret_cast<const f32x4_t*>(p + 4);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[i] = (double)a[i];
            v[4 + i] = (double)b[i];
        }
    }
}

// Whole-call checks of merge_prep's workgroup 0; the status word is written once.
__device__ void merge_validate(const int* __restrict__ kept, const int* __restrict__ offs,
                               const int* __restrict__ coffs, int n_keep,
                               int n_tiles, int n_v, long long ctx_cap, int* __restrict__ status) {
    __shared__ int bad_sh;
    const int tid = threadIdx.x;
    if (tid == 0) bad_sh = 0;
    __syncthreads();
    bool bad = offs[0] != 0 || coffs[0] != 0 || (long long)coffs[n_keep] > ctx_cap;
    for (int i = tid; i < n_keep; i += blockDim.x) {
        const int t = kept[i];
        const int kd = offs[i + 1] - offs[i];
        const int kc = coffs[i + 1] - coffs[i];
        bad |= t < 0 || t >= n_tiles || kd < 0 || kd > n_v || kc < 0 || kc > n_v - kd;
    }
    if (bad) atomicOr(&bad_sh, 1);
    __syncthreads();
    if (tid == 0) *status = bad_sh ? (int)RIFT_ERR_SHAPE : 0;
}

// R (ascending non-dominant tokens) of a tile into lds_r by one wave, from a
// per-token predicate; returns |R| (wave-uniform).
template <typename Pred>
__device__ __forceinline__ int wave_collect(int n_v, int* lds_r, Pred keep) {
    const int lane = threadIdx.x & 63;
    int count = 0;
    for (int base = 0; base < n_v; base += 64) {
        const int t = base + lane;
        const bool k = t < n_v && keep(t);
        const uint64_t m = __ballot(k);
        const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
        if (k) lds_r[count + __popcll(m & below)] = t;
        count += __popcll(m);
    }
    return count;
}

template <bool BF16>
__global__ void __launch_bounds__(256)
merge_prep_kernel(const void* __restrict__ tokens, int n_tiles, int n_v, int d,
                  const int* __restrict__ kept, const int* __restrict__ offs, const int* __restrict__ sel,
                  const int* __restrict__ coffs, int n_keep, long long ctx_cap, int* __restrict__ status,
                  int* __restrict__ grp, int* __restrict__ tgt, double* __restrict__ inv,
                  int* __restrict__ ok) {
    __shared__ int mark[1024];
    __shared__ int rlist[1024];
    __shared__ int n_r_sh, bad_sh;
    const int rho = blockIdx.x;
    const int tid = threadIdx.x;
    if (rho == 0) merge_validate(kept, offs, coffs, n_keep, n_tiles, n_v, ctx_cap, status);
    if (rho >= n_keep) return;
    const int o0 = offs[rho], o1 = offs[rho + 1];
    const int c0 = coffs[rho], c1 = coffs[rho + 1];
    const int tile = kept[rho];
    const int kd = o1 - o0, kc = c1 - c0;
    // this tile's own checks (workgroup 0 reports; a bad tile is skipped)
    if (tile < 0 || tile >= n_tiles || kd < 0 || kd > n_v || kc < 0 || kc > n_v - kd || o0 < 0 ||
        o1 > offs[n_keep] || c0 < 0 || (long long)c1 > ctx_cap) {
        if (tid == 0) ok[rho] = 0;
        return;
    }
    if (tid == 0) bad_sh = 0;
    for (int t = tid; t < n_v; t += blockDim.x) mark[t] = 0;
    __syncthreads();
    for (int k = tid; k < kd; k += blockDim.x) {
        const int t = sel[o0 + k];
        if (t < 0 || t >= n_v) atomicOr(&bad_sh, 1);
        else if (atomicAdd(&mark[t], 1) != 0) atomicOr(&bad_sh, 1);   // duplicate
    }
    __syncthreads();
    if (bad_sh) {
        if (tid == 0) ok[rho] = 0;
        return;
    }
    if (tid < 64) {
        const int n = wave_collect(n_v, rlist, [&](int t) { return mark[t] == 0; });
        if (tid == 0) n_r_sh = n;
    }
    __syncthreads();
    const int n_r = n_r_sh;   // n_v - kd >= kc
    int* g = grp + (size_t)rho * n_v;
    for (int t = tid; t < n_v; t += blockDim.x) g[t] = mark[t] ? -1 : -2;
    __syncthreads();
    for (int j = tid; j < kc; j += blockDim.x) {
        const int t = rlist[(int)(((long long)j * n_r) / kc)];
        tgt[(size_t)rho * n_v + j] = t;
        g[t] = j;
    }
    // inverse norms of the targets: 16 targets per wave, lane r + 16 q
    const int lane = tid & 63, wave = tid >> 6;
    const int r = lane & 15, q = lane >> 4;
    const char* tb = static_cast<const char*>(tokens) + (size_t)tile * n_v * d * (BF16 ? 2 : 4);
    for (int jb = 0; jb < kc; jb += 64) {
        const int j = jb + wave * 16 + r;
        double acc = 0.0;
        if (j < kc) {
            const int t = rlist[(int)(((long long)j * n_r) / kc)];
            for (int s = 0; s < d / 32; ++s) {
                double v[8];
                load8<BF16>(tb, (size_t)t * d + 32 * s + 8 * q, v);
#pragma unroll
                for (int e = 0; e < 8; ++e) acc = fma(v[e], v[e], acc);
            }
        }
        double n2 = acc + __shfl_xor(acc, 32);   // (a0 + a2), (a1 + a3)
        n2 = n2 + __shfl_xor(n2, 16);
        if (j < kc && q == 0) inv[(size_t)rho * n_v + j] = (n2 == 0.0) ? 0.0 : 1.0 / sqrt(n2);
    }
    if (tid == 0) ok[rho] = 1;
}

template <bool BF16>
__global__ void __launch_bounds__(256)
merge_assign_kernel(const void* __restrict__ tokens, int n_v, int d, const int* __restrict__ kept,
                    const int* __restrict__ coffs, int n_keep, int* __restrict__ grp,
                    const int* __restrict__ tgt, const double* __restrict__ inv, const int* __restrict__ ok) {
    __shared__ int rlist[1024];
    __shared__ int n_r_sh;
    __shared__ __align__(16) char tslice[kTB * kDC * 4];   // target block slice (bf16 or f32)
    const int rho = blockIdx.y;
    if (rho >= n_keep || !ok[rho]) return;
    const int kc = coffs[rho + 1] - coffs[rho];
    if (kc < 2) return;   // none, or everything goes to target 0 (set by merge_mean)
    const int tid = threadIdx.x;
    const int* gt = grp + (size_t)rho * n_v;
    if (tid < 64) {
        const int n = wave_collect(n_v, rlist, [&](int t) { return gt[t] != -1; });
        if (tid == 0) n_r_sh = n;
    }
    __syncthreads();
    const int n_r = n_r_sh;
    const int chunk0 = blockIdx.x * 64;
    if (chunk0 >= n_r) return;
    const int lane = tid & 63, wave = tid >> 6;
    const int r16 = lane & 15, q = lane >> 4;
    const int ri = chunk0 + wave * 16 + r16;   // this group's position in R
    const int t_mine = ri < n_r ? rlist[ri] : -1;
    const bool active = t_mine >= 0 && gt[t_mine] == -2;
    const int tile = kept[rho];
    constexpr int EB = BF16 ? 2 : 4;
    const char* tb = static_cast<const char*>(tokens) + (size_t)tile * n_v * d * EB;
    const int* tg = tgt + (size_t)rho * n_v;
    const double* iv = inv + (size_t)rho * n_v;
    double best = 0.0;
    int best_j = -1;
    for (int j0 = 0; j0 < kc; j0 += kTB) {
        const int nb = kc - j0 < kTB ? kc - j0 : kTB;
        double acc[kTB];
#pragma unroll
        for (int k = 0; k < kTB; ++k) acc[k] = 0.0;
        for (int e0 = 0; e0 < d; e0 += kDC) {
            const int ne = d - e0 < kDC ? d - e0 : kDC;   // multiple of 32
            __syncthreads();
            // stage targets [j0, j0 + nb) x elements [e0, e0 + ne) in 16-byte words
            const int wpr = ne * EB / 16;
            for (int w = tid; w < nb * wpr; w += blockDim.x) {
                const int jj = w / wpr, c = w % wpr;
                const int t = tg[j0 + jj];
                *reinterpret_cast<u32x4_t*>(tslice + (size_t)jj * kDC * EB + c * 16) =
                    *reinterpret_cast<const u32x4_t*>(tb + ((size_t)t * d + e0) * EB + c * 16);
            }
            __syncthreads();
            if (active) {
                for (int s = 0; s < ne / 32; ++s) {
                    double x[8];
                    load8<BF16>(tb, (size_t)t_mine * d + e0 + 32 * s + 8 * q, x);
#pragma unroll
                    for (int k = 0; k < kTB; ++k) {
                        if (k < nb) {
                            double y[8];
                            load8<BF16>(tslice + (size_t)k * kDC * EB, 32 * s + 8 * q, y);
#pragma unroll
                            for (int e = 0; e < 8; ++e) acc[k] = fma(x[e], y[e], acc[k]);
                        }
                    }
                }
            }
        }
        // fold the four granule classes, score, running arg-max (ties to the lower j)
#pragma unroll
        for (int k = 0; k < kTB; ++k) {
            double gsum = acc[k] + __shfl_xor(acc[k], 32);
            gsum = gsum + __shfl_xor(gsum, 16);
            if (k < nb) {
                const double a = gsum * iv[j0 + k];
                if (best_j < 0 || a > best) {
                    best = a;
                    best_j = j0 + k;
                }
            }
        }
    }
    if (active && q == 0) grp[(size_t)rho * n_v + t_mine] = best_j;
}

template <bool BF16>
__global__ void __launch_bounds__(256)
merge_mean_kernel(const void* __restrict__ tokens, int n_v, int d, const int* __restrict__ kept,
                  const int* __restrict__ coffs, int n_keep, const int* __restrict__ grp,
                  const int* __restrict__ ok, void* __restrict__ ctx_rows, int* __restrict__ status) {
    __shared__ int members[1024];
    __shared__ int n_mem_sh;
    __shared__ int any_bad;
    const long long row = blockIdx.x;
    if (row == 0) {
        if (threadIdx.x == 0) any_bad = 0;
        __syncthreads();
        for (int i = threadIdx.x; i < n_keep; i += blockDim.x)
            if (!ok[i]) atomicOr(&any_bad, 1);
        __syncthreads();
        if (threadIdx.x == 0 && any_bad) *status = (int)RIFT_ERR_SHAPE;
    }
    if (n_keep <= 0 || row >= coffs[n_keep]) return;
    // the tile whose contextual rows hold this row: largest rho with coffs[rho] <= row
    int lo = 0, hi = n_keep - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (coffs[mid] <= row) lo = mid; else hi = mid - 1;
    }
    const int rho = lo;
    if (!ok[rho]) return;
    const int kc = coffs[rho + 1] - coffs[rho];
    const int j = (int)(row - coffs[rho]);
    if (j < 0 || j >= kc) return;
    const int tid = threadIdx.x;
    const int* gt = grp + (size_t)rho * n_v;
    if (tid < 64) {
        // with one contextual token every remaining token belongs to it
        const int n = wave_collect(n_v, members, [&](int t) {
            const int gv = gt[t];
            return kc == 1 ? gv != -1 : gv == j;
        });
        if (tid == 0) n_mem_sh = n;
    }
    __syncthreads();
    const int n_mem = n_mem_sh;
    constexpr int EB = BF16 ? 2 : 4;
    const char* tb = static_cast<const char*>(tokens) + (size_t)kept[rho] * n_v * d * EB;
    const double cnt = (double)n_mem;
    for (int e0 = tid * 8; e0 < d; e0 += blockDim.x * 8) {
        double acc[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = 0.0;
        for (int m = 0; m < n_mem; ++m) {
            double v[8];
            load8<BF16>(tb, (size_t)members[m] * d + e0, v);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] = acc[e] + v[e];
        }
        float f[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) f[e] = (float)(acc[e] / cnt);
        if constexpr (BF16) {
            u32x4_t w;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                w[i] = (uint32_t)f32_to_bf16(f[2 * i]) | ((uint32_t)f32_to_bf16(f[2 * i + 1]) << 16);
            *reinterpret_cast<u32x4_t*>(static_cast<bf16_t*>(ctx_rows) + (size_t)row * d + e0) = w;
        } else {
            float* o = static_cast<float*>(ctx_rows) + (size_t)row * d + e0;
            *reinterpret_cast<f32x4_t*>(o) = f32x4_t{f[0], f[1], f[2], f[3]};
            *reinterpret_cast<f32x4_t*>(o + 4) = f32x4_t{f[4], f[5], f[6], f[7]};
        }
    }
}

}  // namespace

hipError_t launch_merge(const void* tokens, bool bf16, int n_tiles, int n_v, int d, const int* kept,
                        const int* offs, const int* sel, const int* coffs, int n_keep, void* ctx_rows,
                        long long ctx_cap, int* status, int* grp, int* tgt, double* inv, int* ok,
                        hipStream_t st) {
    const unsigned gp = (unsigned)(n_keep > 0 ? n_keep : 1);
    if (bf16)
        hipLaunchKernelGGL(merge_prep_kernel<true>, dim3(gp), dim3(256), 0, st, tokens, n_tiles, n_v, d, kept,
                           offs, sel, coffs, n_keep, ctx_cap, status, grp, tgt, inv, ok);
    else
        hipLaunchKernelGGL(merge_prep_kernel<false>, dim3(gp), dim3(256), 0, st, tokens, n_tiles, n_v, d, kept,
                           offs, sel, coffs, n_keep, ctx_cap, status, grp, tgt, inv, ok);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (n_keep > 0 && ctx_cap > 0) {
        const dim3 ga((unsigned)((n_v + 63) / 64), (unsigned)n_keep);
        if (bf16)
            hipLaunchKernelGGL(merge_assign_kernel<true>, ga, dim3(256), 0, st, tokens, n_v, d, kept, coffs,
                               n_keep, grp, tgt, inv, ok);
        else
            hipLaunchKernelGGL(merge_assign_kernel<false>, ga, dim3(256), 0, st, tokens, n_v, d, kept, coffs,
                               n_keep, grp, tgt, inv, ok);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    // at least one workgroup: its workgroup 0 finishes the status word
    const unsigned gm = (unsigned)(ctx_cap > 0 ? ctx_cap : 1);
    if (bf16)
        hipLaunchKernelGGL(merge_mean_kernel<true>, dim3(gm), dim3(256), 0, st, tokens, n_v, d, kept, coffs,
                           n_keep, grp, ok, ctx_rows, status);
    else
        hipLaunchKernelGGL(merge_mean_kernel<false>, dim3(gm), dim3(256), 0, st, tokens, n_v, d, kept, coffs,
                           n_keep, grp, ok, ctx_rows, status);
    return hipGetLastError();
}

}  // namespace rift
