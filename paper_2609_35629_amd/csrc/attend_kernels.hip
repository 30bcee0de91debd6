// Split-K attention over the read plan, and the split merge.
//
// k_attend  eq. method-estimate in log space: every row read gets the logit
//           w_{h,i} = scale q_h.k_i - log c_{g(i),h} for each query head h of
//           the KV head (-inf when h did not select the team; no correction
//           for suffix rows and on the dense path), and an online softmax
//           accumulates (m, l, acc) per head.  The rows of one KV head are
//           split into n_split equal ranges over [union rows ; suffix rows];
//           each workgroup owns one range and writes one partial per head.
//           The query heads sharing the KV head share every K/V row load.
// k_merge   rescales the partials of a head to a common maximum and divides
//           the weighted value sum by the mass.
//
// Inside a workgroup: 16 lanes per K/V row, each lane owns d/16 consecutive
// dimensions (one 16-byte load per row and lane for bf16 at d = 128); the 16
// row groups of the workgroup take rows round-robin.  Exponentials are base 2
// with log2(e) folded into the query and the corrections.
#include <math.h>

#include "common.h"
#include "internal.h"

namespace santapp {

namespace {

constexpr int kAttThreads = 256;
constexpr int kAttWaves = kAttThreads / kWave;
constexpr int kAttGroups = kAttThreads / 16;
constexpr int kTileRows = kAttThreads;  // rows described per staging pass
constexpr int kTileTeams = kTileRows + 1;
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kSlotSuffix = -2;
constexpr int kSlotPlain = -1;

template <typename T, int DPL>
struct RowChunk;

template <>
struct RowChunk<bf16_t, 8> {  // d = 128: 8 bf16 = 16 bytes per lane
    static __device__ __forceinline__ void load(const bf16_t* p, float* x) {
        const uint4 u = *reinterpret_cast<const uint4*>(p);
        x[0] = bf16lo(u.x); x[1] = bf16hi(u.x); x[2] = bf16lo(u.y); x[3] = bf16hi(u.y);
        x[4] = bf16lo(u.z); x[5] = bf16hi(u.z); x[6] = bf16lo(u.w); x[7] = bf16hi(u.w);
    }
};

template <>
struct RowChunk<bf16_t, 4> {  // d = 64
    static __device__ __forceinline__ void load(const bf16_t* p, float* x) {
        const uint2 u = *reinterpret_cast<const uint2*>(p);
        x[0] = bf16lo(u.x); x[1] = bf16hi(u.x); x[2] = bf16lo(u.y); x[3] = bf16hi(u.y);
    }
};

template <>
struct RowChunk<float, 8> {
    static __device__ __forceinline__ void load(const float* p, float* x) {
        const float4 a = *reinterpret_cast<const float4*>(p);
        const float4 c = *reinterpret_cast<const float4*>(p + 4);
        x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
        x[4] = c.x; x[5] = c.y; x[6] = c.z; x[7] = c.w;
    }
};

template <>
struct RowChunk<float, 4> {
    static __device__ __forceinline__ void load(const float* p, float* x) {
        const float4 a = *reinterpret_cast<const float4*>(p);
        x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    }
};

// Scale factor of a state with maximum m when rebased to mn (-inf = empty).
__device__ __forceinline__ float rebase(float m, float mn) {
    return (m == -INFINITY) ? 0.f : exp2f(m - mn);
}

template <typename T, int D, int G, bool DENSE>
__global__ __launch_bounds__(kAttThreads) void k_attend(
    const T* __restrict__ K, const T* __restrict__ V, const T* __restrict__ sK,
    const T* __restrict__ sV, const float* __restrict__ q, int N, int T_suf, int M, int Hkv,
    int Hq, int Greal, float scale_log2, int n_split, const int* __restrict__ hdr,
    const int* __restrict__ ubeg, const int* __restrict__ urs, const float* __restrict__ ulogc,
    const int* __restrict__ split_team, float* __restrict__ part_o, float* __restrict__ part_ml) {
    constexpr int DPL = D / 16;
    __shared__ int s_src[kTileRows];
    __shared__ int s_slot[kTileRows];
    __shared__ int s_trs[kTileTeams + 1];
    __shared__ int s_tbeg[kTileTeams];
    __shared__ float s_tlc[kTileTeams][G];
    __shared__ float s_m[kAttWaves][G];
    __shared__ float s_l[kAttWaves][G];
    __shared__ float s_o[kAttWaves][G][D];

    const int s = blockIdx.x;
    const int bh = blockIdx.y;
    const int b = bh / Hkv, kv = bh - b * Hkv;
    const int tid = threadIdx.x, grp = tid >> 4, sub = tid & 15;
    const int lane = lane_id(), w = wave_id();

    int rows_u, U = 0;
    if (DENSE) {
        rows_u = N;
    } else {
        U = hdr[bh * 4 + 0];
        rows_u = hdr[bh * 4 + 1];
    }
    const int total = rows_u + T_suf;
    const int L = (total + n_split - 1) / n_split;
    const int r0 = min(s * L, total), r1 = min(r0 + L, total);

    // the G query heads of this KV head, this lane's dimensions, in log2 units
    float qr[G][DPL];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        const int hq = kv * Greal + h;
#pragma unroll
        for (int e = 0; e < DPL; ++e)
            qr[h][e] = (h < Greal)
                           ? q[(static_cast<size_t>(b) * Hq + hq) * D + sub * DPL + e] * scale_log2
                           : 0.f;
    }
    float m[G], l[G], o[G][DPL];
#pragma unroll
    for (int h = 0; h < G; ++h) {
        m[h] = -INFINITY;
        l[h] = 0.f;
#pragma unroll
        for (int e = 0; e < DPL; ++e) o[h][e] = 0.f;
    }

    const T* Kb = K + static_cast<size_t>(bh) * N * D;
    const T* Vb = V + static_cast<size_t>(bh) * N * D;
    const T* sKb = sK + static_cast<size_t>(bh) * T_suf * D;
    const T* sVb = sV + static_cast<size_t>(bh) * T_suf * D;
    const int* ursb = urs + static_cast<size_t>(bh) * (M + 1);
    const int* ubegb = ubeg + static_cast<size_t>(bh) * M;
    const float* ulcb = ulogc + static_cast<size_t>(bh) * M * kLogcStride;
    int t0 = DENSE ? 0 : split_team[static_cast<size_t>(bh) * n_split + s];

    for (int tile = r0; tile < r1; tile += kTileRows) {
        const int nrows = min(kTileRows, r1 - tile);
        const bool has_union = !DENSE && tile < rows_u;
        if (has_union) {
            // teams t0 .. t0 + kTileRows hold every union row of this tile
            for (int j = tid; j <= kTileTeams; j += kAttThreads) {
                const int t = t0 + j;
                s_trs[j] = (t <= U) ? ursb[t] : 0x7fffffff;
            }
            for (int j = tid; j < kTileTeams; j += kAttThreads) {
                const int t = t0 + j;
                if (t < U) {
                    s_tbeg[j] = ubegb[t];
#pragma unroll
                    for (int h = 0; h < G; ++h) s_tlc[j][h] = ulcb[t * kLogcStride + h] * kLog2e;
                }
            }
            __syncthreads();
        }
        if (tid < nrows) {
            const int r = tile + tid;
            int src, slot;
            if (r < rows_u) {
                if (DENSE) {
                    src = r;
                    slot = kSlotPlain;
                } else {
                    int lo = 0, hi = min(kTileTeams, U - t0) - 1;  // largest j: s_trs[j] <= r
                    while (lo < hi) {
                        const int mid = (lo + hi + 1) >> 1;
                        if (s_trs[mid] <= r)
                            lo = mid;
                        else
                            hi = mid - 1;
                    }
                    src = s_tbeg[lo] + (r - s_trs[lo]);
                    slot = lo;
                }
            } else {
                src = r - rows_u;
                slot = kSlotSuffix;
            }
            s_src[tid] = src;
            s_slot[tid] = slot;
        }
        __syncthreads();

        for (int i = grp; i < nrows; i += kAttGroups) {
            const int src = s_src[i], slot = s_slot[i];
            const T* kp = (slot == kSlotSuffix) ? sKb : Kb;
            const T* vp = (slot == kSlotSuffix) ? sVb : Vb;
            float kx[DPL], vx[DPL];
            RowChunk<T, DPL>::load(kp + static_cast<size_t>(src) * D + sub * DPL, kx);
            RowChunk<T, DPL>::load(vp + static_cast<size_t>(src) * D + sub * DPL, vx);
            float sc[G];
#pragma unroll
            for (int h = 0; h < G; ++h) {
                float a = 0.f;
#pragma unroll
                for (int e = 0; e < DPL; ++e) a = fmaf(qr[h][e], kx[e], a);
                sc[h] = a;
            }
#pragma unroll
            for (int h = 0; h < G; ++h) {
#pragma unroll
                for (int off = 8; off > 0; off >>= 1) sc[h] += __shfl_xor(sc[h], off, 16);
            }
#pragma unroll
            for (int h = 0; h < G; ++h) {
                const float wv = (slot >= 0) ? sc[h] - s_tlc[slot][h] : sc[h];
                const float mn = fmaxf(m[h], wv);
                if (mn == -INFINITY) continue;  // nothing accumulated and nothing to add
                const float a = rebase(m[h], mn);
                const float p = exp2f(wv - mn);  // 0 for a masked head
                l[h] = l[h] * a + p;
#pragma unroll
                for (int e = 0; e < DPL; ++e) o[h][e] = fmaf(p, vx[e], o[h][e] * a);
                m[h] = mn;
            }
        }
        __syncthreads();
        if (has_union && nrows == kTileRows) {
            const int last = s_slot[kTileRows - 1];
            if (last >= 0) t0 += last;  // team of the tile's last row
        }
    }

    // merge the four row groups of each wave, then the waves
#pragma unroll
    for (int off = 16; off < kWave; off <<= 1) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
            const float m2 = __shfl_xor(m[h], off);
            const float l2 = __shfl_xor(l[h], off);
            float o2[DPL];
#pragma unroll
            for (int e = 0; e < DPL; ++e) o2[e] = __shfl_xor(o[h][e], off);
            const float mn = fmaxf(m[h], m2);
            const float a = rebase(m[h], mn), c = rebase(m2, mn);
            l[h] = l[h] * a + l2 * c;
#pragma unroll
            for (int e = 0; e < DPL; ++e) o[h][e] = o[h][e] * a + o2[e] * c;
            m[h] = mn;
        }
    }
    if (lane < 16) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
#pragma unroll
            for (int e = 0; e < DPL; ++e) s_o[w][h][sub * DPL + e] = o[h][e];
            if (lane == 0) {
                s_m[w][h] = m[h];
                s_l[w][h] = l[h];
            }
        }
    }
    __syncthreads();
    for (int idx = tid; idx < Greal * D; idx += kAttThreads) {
        const int h = idx / D, j = idx - h * D;
        float mx = -INFINITY;
#pragma unroll
        for (int v = 0; v < kAttWaves; ++v) mx = fmaxf(mx, s_m[v][h]);
        float lsum = 0.f, osum = 0.f;
#pragma unroll
        for (int v = 0; v < kAttWaves; ++v) {
            const float a = rebase(s_m[v][h], mx);
            lsum += s_l[v][h] * a;
            osum += s_o[v][h][j] * a;
        }
        const size_t pidx = (static_cast<size_t>(b) * Hq + kv * Greal + h) * n_split + s;
        part_o[pidx * D + j] = osum;
        if (j == 0) {
            part_ml[pidx * 2 + 0] = mx;
            part_ml[pidx * 2 + 1] = lsum;
        }
    }
}

__global__ void k_merge(const float* __restrict__ part_o, const float* __restrict__ part_ml,
                        int n_split, int D, float* __restrict__ out) {
    const size_t bhq = blockIdx.x;
    const int j = threadIdx.x;
    const float* ml = part_ml + bhq * n_split * 2;
    float mx = -INFINITY;
    for (int s = 0; s < n_split; ++s) mx = fmaxf(mx, ml[2 * s]);
    float lsum = 0.f, osum = 0.f;
    for (int s = 0; s < n_split; ++s) {
        const float a = rebase(ml[2 * s], mx);
        lsum += ml[2 * s + 1] * a;
        osum += part_o[(bhq * n_split + s) * D + j] * a;
    }
    out[bhq * D + j] = osum / lsum;
}

__global__ void k_zero(uint4* __restrict__ p, size_t n16, unsigned char* __restrict__ tail,
                       int ntail) {
    const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
    for (size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; i < n16; i += stride)
        p[i] = make_uint4(0, 0, 0, 0);
    if (blockIdx.x == 0 && static_cast<int>(threadIdx.x) < ntail) tail[threadIdx.x] = 0;
}

template <typename T, int D, int G>
hipError_t attend_g(const AttendArgs& a, hipStream_t s) {
    const dim3 grid(a.n_split, a.B * a.Hkv);
    const float sl2 = a.scale * kLog2e;
    const T* K = static_cast<const T*>(a.K);
    const T* V = static_cast<const T*>(a.V);
    const T* sK = static_cast<const T*>(a.sK);
    const T* sV = static_cast<const T*>(a.sV);
    if (a.dense) {
        k_attend<T, D, G, true><<<grid, kAttThreads, 0, s>>>(
            K, V, sK, sV, a.q, a.N, a.T, 0, a.Hkv, a.Hq, a.G, sl2, a.n_split, nullptr, nullptr,
            nullptr, nullptr, nullptr, a.part_o, a.part_ml);
    } else {
        const DecodeLayout& L = *a.lay;
        k_attend<T, D, G, false><<<grid, kAttThreads, 0, s>>>(
            K, V, sK, sV, a.q, a.N, a.T, a.M, a.Hkv, a.Hq, a.G, sl2, a.n_split,
            reinterpret_cast<const int*>(a.ws + L.hdr), reinterpret_cast<const int*>(a.ws + L.ubeg),
            reinterpret_cast<const int*>(a.ws + L.urs),
            reinterpret_cast<const float*>(a.ws + L.ulogc),
            reinterpret_cast<const int*>(a.ws + L.split), a.part_o, a.part_ml);
    }
    return hipGetLastError();
}

template <typename T, int D>
hipError_t attend_d(const AttendArgs& a, hipStream_t s) {
    switch (a.G) {
        case 1: return attend_g<T, D, 1>(a, s);
        case 2: return attend_g<T, D, 2>(a, s);
        case 3:
        case 4: return attend_g<T, D, 4>(a, s);
        case 5:
        case 6:
        case 7: return attend_g<T, D, 7>(a, s);
        case 8: return attend_g<T, D, 8>(a, s);
        default: return hipErrorInvalidValue;
    }
}

template <typename T>
hipError_t attend_t(const AttendArgs& a, hipStream_t s) {
    switch (a.d) {
        case 64: return attend_d<T, 64>(a, s);
        case 128: return attend_d<T, 128>(a, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_attend(const AttendArgs& a, hipStream_t s) {
    return a.dtype == SANTAPP_BF16 ? attend_t<bf16_t>(a, s) : attend_t<float>(a, s);
}

hipError_t launch_merge(const AttendArgs& a, hipStream_t s) {
    k_merge<<<a.B * a.Hq, a.d, 0, s>>>(a.part_o, a.part_ml, a.n_split, a.d, a.out);
    return hipGetLastError();
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s) {
    const size_t n16 = bytes / 16;
    const int ntail = static_cast<int>(bytes - n16 * 16);
    const size_t want = (n16 + 255) / 256;
    const unsigned blocks = static_cast<unsigned>(want == 0 ? 1 : (want < 4096 ? want : 4096));
    k_zero<<<blocks, 256, 0, s>>>(static_cast<uint4*>(p), n16,
                                  static_cast<unsigned char*>(p) + n16 * 16, ntail);
    return hipGetLastError();
}

}  // namespace santapp
