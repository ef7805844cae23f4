// Forward of one batch: pooled embedding-bag lookup over the two-tier store.
//
// Order of work on the stream (dedup and probe live in dedup.hip):
//   k_fwd_prep   validate bag offsets, record each table's index range
//   k_mark / count / scan / emit(FORWARD)   distinct rows, sorted; map probe
//   k_fwd_src    per index: where its row lives (slot or staging row, and
//                that row's device address), through the rank of the row
//                among the distinct rows
//   k_fetch      ZERO_COPY: copy each distinct missing row once from pinned
//                host memory to HBM staging (GPU reads over the host link)
//   k_pool       per bag, sum of its rows in fp32 (Sec. II, pooling by sum)
//   k_fwd_finalize  publish the counters
#include <type_traits>

#include <hip/hip_ext.h>

#include "launch.h"

namespace recmg {

__global__ void __launch_bounds__(kBlock) k_fwd_prep(DGlobal g, const int64_t *__restrict__ offsets, int32_t B,
                                                     int64_t n) {
    const int64_t nb = (int64_t)g.T * B;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < nb && offsets[i] > offsets[i + 1]) atomicOr(g.err, ERR_OFFSETS);
    if (i == 0 && (offsets[0] != 0 || offsets[nb] != n)) atomicOr(g.err, ERR_OFFSETS);
    if (i <= g.T) g.tstart[i] = offsets[i * (int64_t)B];
    if (i < g.T) {
        TState &st = g.st[i];
        st.ucount = 0;
        st.mcount = 0;
        st.hits = 0;
        st.hits_pf = 0;
        st.covered = 0;
    }
}

// Coverage (Eq. coverage): how many distinct rows of the last placement's
// prefetch list (PU, still in place) this batch touches.  A row is in the
// batch iff its rank word carries this forward's stamp and its bit.
__global__ void __launch_bounds__(kBlock) k_fwd_cover(DGlobal g, int32_t stamp, int64_t np) {
    if (*g.err) return;
    __shared__ int64_t s_pstart[RECMG_MAX_TABLES + 1];
    __shared__ int32_t s_pc[RECMG_MAX_TABLES];
    __shared__ int s_cov[RECMG_MAX_TABLES];
    for (int t = threadIdx.x; t <= g.T; t += blockDim.x) {
        s_pstart[t] = g.pstart[t];
        if (t < g.T) {
            s_pc[t] = g.st[t].pcount;
            s_cov[t] = 0;
        }
    }
    __syncthreads();
    int64_t lo, hi;
    block_share(np, &lo, &hi);
    for (int64_t base = lo; base < hi; base += blockDim.x) {  // block-uniform
        const int64_t i = base + threadIdx.x;
        int t = 0;
        bool hit = false;
        if (i < hi) {
            t = find_seg(s_pstart, g.T, i);
            if (i - s_pstart[t] < s_pc[t]) {
                const DTable &tb = g.tabs[t];
                const uint32_t pos = bm_pos(tb, g.PU[i]);
                const uint4 rk = tb.rank[pos >> 5];
                hit = (int32_t)rk.z == stamp && (rk.y & (1u << (pos & 31)));
            }
        }
        wave_count_lds(hit, t, s_cov);  // counts only
    }
    __syncthreads();
    for (int t = threadIdx.x; t < g.T; t += blockDim.x)
        if (s_cov[t]) atomicAdd(&g.st[t].covered, s_cov[t]);
}

// Cache probe of every distinct row (row -> slot map, or a scan of the row's
// set in a set-associative table): hits are stamped and
// counted, misses are numbered (their staging row).  One thread per slot of
// the index space; table t's distinct rows occupy [tstart[t], + ucount).
__global__ void __launch_bounds__(kBlock) k_fwd_probe(DGlobal g, int32_t stamp, int64_t n) {
    if (*g.err) return;
    __shared__ int64_t s_start[RECMG_MAX_TABLES + 1];
    __shared__ int32_t s_uc[RECMG_MAX_TABLES];
    __shared__ int s_hits[RECMG_MAX_TABLES], s_hits_pf[RECMG_MAX_TABLES];
    for (int t = threadIdx.x; t <= g.T; t += blockDim.x) {
        s_start[t] = g.tstart[t];
        if (t < g.T) {
            s_uc[t] = g.st[t].ucount;
            s_hits[t] = 0;
            s_hits_pf[t] = 0;
        }
    }
    __syncthreads();
    int32_t *mcount0 = &g.st[0].mcount;
    const int stride_st = (int)(sizeof(TState) / 4);
    int64_t lo, hi;
    block_share(n, &lo, &hi);
    for (int64_t base = lo; base < hi; base += blockDim.x) {  // block-uniform
        const int64_t i = base + threadIdx.x;
        int t = 0;
        bool miss = false, valid = false, hit = false, hit_pf = false;
        int32_t row = 0;
        if (i < hi) {
            t = find_seg(s_start, g.T, i);
            valid = i - s_start[t] < s_uc[t];
        }
        if (valid) {
            const DTable &tb = g.tabs[t];
            row = g.U[i];
            const int32_t slot = find_slot(tb, row);
            if (slot >= 0) {
                g.slotU[i] = slot;
                tb.slot_touch[slot] = stamp;
                hit = true;
                hit_pf = (tb.slot_flags[slot] & F_PF) != 0;
            } else {
                miss = true;
            }
        }
        wave_count_lds(hit, t, s_hits);  // counts only
        wave_count_lds(hit_pf, t, s_hits_pf);
        const int32_t m = wave_append(miss, t, mcount0, stride_st);
        if (miss) {
            const int64_t at = s_start[t] + m;
            g.slotU[i] = -(m + 1);
            g.M[at] = row;
            g.mflags[at] = 0;
            g.mcbit[at] = 0;
        }
    }
    __syncthreads();
    for (int t = threadIdx.x; t < g.T; t += blockDim.x) {
        if (s_hits[t]) atomicAdd(&g.st[t].hits, s_hits[t]);
        if (s_hits_pf[t]) atomicAdd(&g.st[t].hits_pf, s_hits_pf[t]);
    }
}

// inverse map and data location of every index
__global__ void __launch_bounds__(kBlock) k_fwd_src(DGlobal g, const int32_t *__restrict__ indices, int64_t n) {
    if (*g.err) return;
    __shared__ int64_t s_start[RECMG_MAX_TABLES + 1];
    __shared__ const uint4 *s_rank[RECMG_MAX_TABLES];
    __shared__ const char *s_pool[RECMG_MAX_TABLES];
    __shared__ int32_t s_rb[RECMG_MAX_TABLES], s_ns[RECMG_MAX_TABLES], s_qb[RECMG_MAX_TABLES];
    for (int t = threadIdx.x; t <= g.T; t += blockDim.x) {
        s_start[t] = g.tstart[t];
        if (t < g.T) {
            s_rank[t] = g.tabs[t].rank;
            s_pool[t] = g.tabs[t].pool;
            s_rb[t] = g.tabs[t].row_bytes;
            s_ns[t] = g.tabs[t].nsets;
            s_qb[t] = g.tabs[t].qbits;
        }
    }
    __syncthreads();
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const int t = find_seg(s_start, g.T, i);
        const uint32_t pos = bm_pos(s_ns[t], s_qb[t], indices[i]);
        const uint4 rk = s_rank[t][pos >> 5];
        const int32_t u = (int32_t)rk.x + __popc(rk.y & ((1u << (pos & 31)) - 1u));
        const int32_t sl = g.slotU[s_start[t] + u];
        g.src[i] = sl;
        g.raddr[i] = sl >= 0 ? (uint64_t)(s_pool[t] + (int64_t)sl * s_rb[t])
                             : (uint64_t)(g.staging + (s_start[t] - (int64_t)sl - 1) * g.stage_stride);
    }
}

// ----------------------------------------------------------------- miss fetch

// ZERO_COPY miss fetch: each distinct miss of a zero-copy table is read once
// from pinned host memory (device-visible mapping) and written to its staging
// row (STAGED tables' misses are staged by the host).
__global__ void __launch_bounds__(kBlock) k_fetch(DGlobal g) {
    if (*g.err) return;
    __shared__ int32_t s_cnt[RECMG_MAX_TABLES];
    for (int t = threadIdx.x; t < g.T; t += blockDim.x) s_cnt[t] = g.tabs[t].staged ? 0 : g.st[t].mcount;
    __syncthreads();
    copy_flat(
        g, s_cnt, gridDim.x,
        [&](int t, const DTable &tb, int64_t j) {
            return tb.host + (int64_t)g.M[g.tstart[t] + j] * tb.row_bytes;
        },
        [&](int t, const DTable &tb, int64_t j) { return g.staging + (g.tstart[t] + j) * g.stage_stride; });
}

// ----------------------------------------------------------------- pooling

template <int DT>
struct Elem;
template <>
struct Elem<RECMG_F32> {
    static constexpr int bytes = 4;
    __device__ static float widen(uint32_t x) { return __builtin_bit_cast(float, x); }
};
template <>
struct Elem<RECMG_F16> {
    static constexpr int bytes = 2;
    __device__ static float widen(uint32_t x) { return f16_to_f32(x & 0xffffu); }
};
template <>
struct Elem<RECMG_BF16> {
    static constexpr int bytes = 2;
    __device__ static float widen(uint32_t x) { return bf16_to_f32(x & 0xffffu); }
};

// 16-byte vector of elements -> VE floats added into acc
template <int DT>
__device__ __forceinline__ void accum_vec(float *acc, const uint4 v) {
    if constexpr (DT == RECMG_F32) {
        acc[0] += __builtin_bit_cast(float, v.x);
        acc[1] += __builtin_bit_cast(float, v.y);
        acc[2] += __builtin_bit_cast(float, v.z);
        acc[3] += __builtin_bit_cast(float, v.w);
    } else {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if constexpr (DT == RECMG_BF16) {
                acc[2 * k] += __builtin_bit_cast(float, w[k] << 16);
                acc[2 * k + 1] += __builtin_bit_cast(float, w[k] & 0xffff0000u);
            } else {
                acc[2 * k] += f16_to_f32(w[k] & 0xffffu);
                acc[2 * k + 1] += f16_to_f32(w[k] >> 16);
            }
        }
    }
}

template <int DT, bool VEC>
struct Lane {
    static constexpr int VE = VEC ? 16 / Elem<DT>::bytes : 1;
    using V = typename std::conditional<VEC, uint4, typename std::conditional<Elem<DT>::bytes == 4, uint32_t,
                                                                               uint16_t>::type>::type;
    __device__ static V load(const char *p) {
        if constexpr (VEC) return gload16(p);
        else if constexpr (Elem<DT>::bytes == 4) return gload4(p);
        else return gload2(p);
    }
    __device__ static void add(float *acc, const V v) {
        if constexpr (VEC) accum_vec<DT>(acc, v);
        else acc[0] += Elem<DT>::widen((uint32_t)v);
    }
};

// One group of G lanes sums one bag.  Lookup p of the bag goes to
// accumulator p mod 4; the four partial sums are combined pairwise at the end.
// The order is fixed per bag, so the result does not depend on which tier
// served each row.  The group keeps up to 16 row loads in flight and loads the
// next chunk of locations while the current chunk's rows are in flight.
template <int DT, bool VEC>
__device__ __forceinline__ void pool_table(const DGlobal &g, const DTable &tb, int t, int32_t B,
                                           const int64_t *__restrict__ offsets, float *__restrict__ out,
                                           int blk_in_table) {
    using L = Lane<DT, VEC>;
    using V = typename L::V;
    constexpr int VE = L::VE;
    constexpr int EB = Elem<DT>::bytes;
#ifndef RECMG_POOL_UNROLL
#define RECMG_POOL_UNROLL 8
#endif
#ifndef RECMG_POOL_UNROLL_HALF
#define RECMG_POOL_UNROLL_HALF 8
#endif
    // row loads in flight per group (fp32 / 2-byte storage): measured best on
    // gfx950, where more depth costs more in occupancy than it gains
    constexpr int UNROLL = EB == 4 ? RECMG_POOL_UNROLL : RECMG_POOL_UNROLL_HALF;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int G = tb.gsz;
    const int gl = lane & (G - 1);
    const int gi = lane / G;
    const int bpw = 64 / G;
    const int j = (blk_in_table * (kBlock / 64) + wave) * bpw + gi;
    if (j >= B) return;
    const int64_t a = offsets[(int64_t)t * B + j], e = offsets[(int64_t)t * B + j + 1];
    const int D = tb.dim;
    const int64_t rb = tb.row_bytes;
    const char *__restrict__ pool = tb.pool;
    const int64_t sstride = g.stage_stride;
    const char *__restrict__ stg = g.staging + g.tstart[t] * sstride;
    const int32_t *__restrict__ src = g.src;
    float *orow = out + (int64_t)B * tb.out_elem_off + (int64_t)j * D;

    for (int ch = 0; ch < tb.nchunk; ++ch) {
        const int e0 = (ch * G + gl) * VE;
        const bool lane_ok = e0 < D;
        const int64_t eoff = lane_ok ? (int64_t)e0 * EB : 0;
        // slot s >= 0: the HBM pool; s < 0: staging row -(s + 1); no branch
        auto row_ptr = [&](int s) -> const char * {
            const bool hit = s >= 0;
            const char *base = hit ? pool : stg;
            const int64_t idx = hit ? s : -(int64_t)s - 1;
            return base + idx * (hit ? rb : sstride) + eoff;
        };
        float acc[4][VE];
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int x = 0; x < VE; ++x) acc[k][x] = 0.f;

        int my = (a + gl < e) ? (int)gload4(src + a + gl) : 0;
        for (int64_t c = a; c < e; c += G) {
            const int n = (int)((e - c) < G ? (e - c) : G);
            const int nxt = (c + G + gl < e) ? (int)gload4(src + c + G + gl) : 0;  // next chunk, in flight meanwhile
            int q = 0;
            for (; q + UNROLL <= n; q += UNROLL) {
                int sv[UNROLL];
#pragma unroll
                for (int u = 0; u < UNROLL; ++u) sv[u] = __shfl(my, q + u, G);
                V v[UNROLL];
#pragma unroll
                for (int u = 0; u < UNROLL; ++u) v[u] = L::load(row_ptr(sv[u]));
#pragma unroll
                for (int u = 0; u < UNROLL; ++u) L::add(acc[u & 3], v[u]);
            }
            for (; q < n; q += 4) {
                int sv[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) sv[u] = __shfl(my, q + u < n ? q + u : q, G);
                V v[4];
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (q + u < n) v[u] = L::load(row_ptr(sv[u]));
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (q + u < n) L::add(acc[u], v[u]);
            }
            my = nxt;
        }
        if (lane_ok) {
            float r[VE];
#pragma unroll
            for (int x = 0; x < VE; ++x) r[x] = (acc[0][x] + acc[1][x]) + (acc[2][x] + acc[3][x]);
            float *o = orow + e0;
            if (VE % 4 == 0 && (((uintptr_t)o) & 15) == 0) {
#pragma unroll
                for (int x = 0; x < VE; x += 4)
                    *reinterpret_cast<float4 *>(o + x) = make_float4(r[x], r[x + 1], r[x + 2], r[x + 3]);
            } else {
#pragma unroll
                for (int x = 0; x < VE; ++x) o[x] = r[x];
            }
        }
    }
}

// Workgroups are dealt round-robin to the 8 XCDs; give each XCD one
// contiguous range of a launch's blocks so a table's hot rows stay in one L2.
__device__ __forceinline__ int xcd_block(int nb) {
#ifndef RECMG_POOL_NO_XCD_MAP
    const int x = (int)blockIdx.x & 7, q = nb >> 3, r = nb & 7;
    return x * q + (x < r ? x : r) + ((int)blockIdx.x >> 3);
#else
    return (int)blockIdx.x;
#endif
}

// Group-per-bag kernel for the tables the wave-per-bag kernel does not take.
// Each launch covers the blocks [boff, boff + nblk) of one class; block lb
// belongs to table btab[k] for the k with bstart[k] <= lb < bstart[k + 1].
template <int DT, bool VEC>
__global__ void __launch_bounds__(kBlock) k_pool(DGlobal g, const int64_t *__restrict__ offsets, int32_t B,
                                                 float *__restrict__ out, const int32_t *__restrict__ bstart,
                                                 const int32_t *__restrict__ btab, int32_t nt, int32_t boff,
                                                 int32_t nblk) {
    if (*g.err) return;
    const int lb = boff + xcd_block(nblk);
    __shared__ int s_k;
    if (threadIdx.x == 0) s_k = find_seg32(bstart, nt, lb);
    __syncthreads();
    const int k = s_k, t = btab[k];
    pool_table<DT, VEC>(g, g.tabs[t], t, B, offsets, out, lb - bstart[k]);
}

// ------------------------------------------------- wave-per-bag pooled sum
//
// One wave sums kWaveBags consecutive bags, one bag at a time.  Each lane
// adds its LW-byte slice of every row; row addresses come from the per-index
// array written by k_fwd_src, so the kernel does no slot or staging lookups.
//   R == 1 (rows of 1024 bytes or whole multiples): all lanes read the same
//     row, so its address is wave-uniform and comes in through scalar loads.
//   R > 1 (shorter rows): the wave splits into R groups of 64 / R lanes that
//     read R different rows per load instruction, group h taking the lookups
//     p with p mod R = h.  Each lane holds one address of a window of 64
//     lookups; a ds_bpermute hands every group its row's address.
// Either way lookup p goes to partial sum p mod 4 and the four are combined
// as (S0 + S1) + (S2 + S3): a fixed order per bag, whichever tier served a row.

template <int LW>
struct WVec;
template <>
struct WVec<4> {
    using V = uint32_t;
    __device__ static void words(const V v, uint32_t *w) { w[0] = v; }
};
template <>
struct WVec<8> {
    using V = u32x2_t;
    __device__ static void words(const V v, uint32_t *w) {
        w[0] = v.x;
        w[1] = v.y;
    }
};
template <>
struct WVec<16> {
    using V = u32x4_t;
    __device__ static void words(const V v, uint32_t *w) {
        w[0] = v.x;
        w[1] = v.y;
        w[2] = v.z;
        w[3] = v.w;
    }
};

// acc + the fp16 value in the low / high half of w: one mixed-precision FMA
// (x * 1 + acc) converts exactly and rounds once, like convert-then-add
__device__ __forceinline__ float add_f16_lo(float acc, uint32_t w) {
    float r;
    asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel_hi:[1,0,0]" : "=v"(r) : "v"(w), "v"(acc));
    return r;
}
__device__ __forceinline__ float add_f16_hi(float acc, uint32_t w) {
    float r;
    asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "=v"(r) : "v"(w), "v"(acc));
    return r;
}

template <int DT, int LW>
__device__ __forceinline__ void wadd(float *acc, const typename WVec<LW>::V v) {
    uint32_t w[LW / 4];
    WVec<LW>::words(v, w);
#pragma unroll
    for (int k = 0; k < LW / 4; ++k) {
        if constexpr (DT == RECMG_F32) {
            acc[k] += __builtin_bit_cast(float, w[k]);
        } else if constexpr (DT == RECMG_BF16) {
            acc[2 * k] += __builtin_bit_cast(float, w[k] << 16);
            acc[2 * k + 1] += __builtin_bit_cast(float, w[k] & 0xffff0000u);
        } else {
            acc[2 * k] = add_f16_lo(acc[2 * k], w[k]);
            acc[2 * k + 1] = add_f16_hi(acc[2 * k + 1], w[k]);
        }
    }
}

// LW-byte load at global address base + off
template <class V>
__device__ __forceinline__ V wload(uint64_t base, uint32_t off) {
    typedef const __attribute__((address_space(1))) char gchar;
    return *(const __attribute__((address_space(1))) V *)((gchar *)base + off);
}

// The lane offset is passed through an empty asm in every block of loads so
// that its zero extension is visible where the loads are selected: a uniform
// 64-bit base plus a 32-bit lane offset then becomes the scalar-base form of
// global_load, with no vector address arithmetic at all.
__device__ __forceinline__ uint32_t opaque(uint32_t x) {
    asm volatile("" : "+v"(x));
    return x;
}

// Combine the NA partial sums of each of the R groups in the order
// (S0 + S1) + (S2 + S3) and store the bag's NE floats of this lane (group 0).
template <int NE, int R, int NA>
__device__ __forceinline__ void wstore(float (&acc)[NA][NE], int h, float *o) {
    float r[NE];
#pragma unroll
    for (int x = 0; x < NE; ++x) {
        if constexpr (R == 1) {
            r[x] = (acc[0][x] + acc[1][x]) + (acc[2][x] + acc[3][x]);
        } else if constexpr (R == 2) {
            // group 0 holds S0, S2 and group 1 holds S1, S3
            const float o0 = __shfl_xor(acc[0][x], 32), o1 = __shfl_xor(acc[1][x], 32);
            r[x] = (acc[0][x] + o0) + (acc[1][x] + o1);
        } else {
            // group h holds S_h
            const float s01 = acc[0][x] + __shfl_xor(acc[0][x], 16);
            r[x] = s01 + __shfl_xor(s01, 32);
        }
    }
    if (h != 0) return;
    // a table's output block starts at B * (sum of the earlier dims) floats,
    // so vector stores need a run-time alignment check
    const uintptr_t oa = reinterpret_cast<uintptr_t>(o);
    if (NE % 4 == 0 && (oa & 15) == 0) {
#pragma unroll
        for (int x = 0; x + 3 < NE; x += 4)
            *reinterpret_cast<float4 *>(o + x) = make_float4(r[x], r[x + 1], r[x + 2], r[x + 3]);
    } else if (NE == 2 && (oa & 7) == 0) {
        *reinterpret_cast<float2 *>(o) = make_float2(r[0], r[NE - 1]);
    } else {
#pragma unroll
        for (int x = 0; x < NE; ++x) o[x] = r[x];
    }
}

// the bag offsets of the wave's bags, clamped to the last one present
template <int BPW>
__device__ __forceinline__ void wave_offsets(int64_t (&offs)[BPW + 1], const int64_t *__restrict__ ob, int nbags) {
#pragma unroll
    for (int b = 0; b <= BPW; ++b) offs[b] = ob[b < nbags ? b : nbags];
}

// R == 1.  Software pipeline: the scalar loads of the next block's U row
// addresses (this bag's, else the next non-empty bag's first) are in flight
// while the current block's row loads are.  A block may run past the bag and
// past the batch (the address array has kRaddrPad entries of padding); such
// addresses are never dereferenced.
template <int DT, int LW>
__device__ __forceinline__ void pool_wave_s(const uint64_t *__restrict__ raddr, const int64_t *__restrict__ ob,
                                            int nbags, int wnch, int D, float *__restrict__ obase) {
    using V = typename WVec<LW>::V;
    constexpr int EB = Elem<DT>::bytes, NE = LW / EB;
    constexpr int U = 8;  // rows in flight per wave (8 KB)
    constexpr int BPW = kWaveBags;
    const int lane = threadIdx.x & 63;
    int64_t offs[BPW + 1];
    wave_offsets<BPW>(offs, ob, nbags);
    for (int ch = 0; ch < wnch; ++ch) {
        const uint32_t eoff = (uint32_t)((ch * 64 + lane) * LW);
        uint64_t nx[U];
        // first block of the first non-empty bag after bag b (all indices
        // static, so offs and nx stay in scalar registers)
        auto next_bag_addrs = [&](int b) {
            bool found = false;
#pragma unroll
            for (int b2 = 0; b2 < BPW; ++b2)
                if (b2 > b && !found && b2 < nbags && offs[b2 + 1] > offs[b2]) {
#pragma unroll
                    for (int k = 0; k < U; ++k) nx[k] = raddr[offs[b2] + k];
                    found = true;
                }
        };
        next_bag_addrs(-1);
#pragma unroll
        for (int b = 0; b < BPW; ++b) {
            if (b >= nbags) continue;
            const int64_t a = offs[b];
            const int n = (int)(offs[b + 1] - a);
            float acc[4][NE];
#pragma unroll
            for (int k = 0; k < 4; ++k)
#pragma unroll
                for (int x = 0; x < NE; ++x) acc[k][x] = 0.f;
            int p = 0;
            for (; p + U <= n; p += U) {
                V v[U];
                const uint32_t eo = opaque(eoff);
#pragma unroll
                for (int u = 0; u < U; ++u) v[u] = wload<V>(nx[u], eo);
                // the barrier keeps the next block's scalar loads after the
                // row loads above, so one block of addresses is live at a time
                asm volatile("" ::: "memory");
                if (p + U < n) {
#pragma unroll
                    for (int k = 0; k < U; ++k) nx[k] = raddr[a + p + U + k];
                } else {
                    next_bag_addrs(b);
                }
#pragma unroll
                for (int u = 0; u < U; ++u) wadd<DT, LW>(acc[u & 3], v[u]);
            }
            if (p < n) {
                // partial block, in quads of loads; a lookup past the bag's end
                // re-reads the quad's first row and is not added
                V v[U];
#pragma unroll
                for (int q = 0; q < U; q += 4)
                    if (p + q < n) {
                        const uint32_t eo = opaque(eoff);
#pragma unroll
                        for (int u = q; u < q + 4; ++u) v[u] = wload<V>(p + u < n ? nx[u] : nx[q], eo);
                    }
                asm volatile("" ::: "memory");
                next_bag_addrs(b);
#pragma unroll
                for (int u = 0; u < U; ++u)
                    if (p + u < n) wadd<DT, LW>(acc[u & 3], v[u]);
            }
            wstore<NE, 1, 4>(acc, 0, obase + (int64_t)b * D + ch * 64 * NE + lane * NE);
        }
    }
}

#ifndef RECMG_WPOOL_KB
#define RECMG_WPOOL_KB 8
#endif

// R > 1.  Lane i holds the address of lookup w + i of a window of 64 lookups
// of the bag starting at w (a whole bag when it has at most 64); the next
// window (this bag's, else the next non-empty bag's first) is loaded while
// the current one's rows are read.  Window entries past the bag, and past the
// batch (kRaddrPad entries of padding), are never dereferenced.
template <int DT, int LW, int R>
__device__ __forceinline__ void pool_wave_v(const uint64_t *__restrict__ raddr, const int64_t *__restrict__ ob,
                                            int nbags, int D, float *__restrict__ obase) {
    using V = typename WVec<LW>::V;
    constexpr int EB = Elem<DT>::bytes, NE = LW / EB, GL = 64 / R, NA = 4 / R;
    constexpr int U0 = RECMG_WPOOL_KB * 16 / LW;  // load instructions per sub-block (KB of rows in flight)
    constexpr int U = U0 * R > 64 ? 64 / R : U0;  // a sub-block stays inside its window
    constexpr int UR = U * R;                    // lookups per sub-block, divides 64
    static_assert(64 % UR == 0 && U % NA == 0, "sub-blocks tile a window; slot = u mod NA");
    constexpr int BPW = kWaveBags;
    const int lane = threadIdx.x & 63, h = lane / GL, gl = lane % GL;
    const uint32_t eoff = (uint32_t)(gl * LW);
    int64_t offs[BPW + 1];
    wave_offsets<BPW>(offs, ob, nbags);
    uint64_t wnext = 0;
    auto next_bag_window = [&](int b) {
        bool found = false;
#pragma unroll
        for (int b2 = 0; b2 < BPW; ++b2)
            if (b2 > b && !found && b2 < nbags && offs[b2 + 1] > offs[b2]) {
                wnext = RECMG_GLOBAL(uint64_t, raddr + offs[b2] + lane);
                found = true;
            }
    };
    next_bag_window(-1);
#pragma unroll
    for (int b = 0; b < BPW; ++b) {
        if (b >= nbags) continue;
        const int64_t a = offs[b];
        const int n = (int)(offs[b + 1] - a);
        float acc[NA][NE];
#pragma unroll
        for (int k = 0; k < NA; ++k)
#pragma unroll
            for (int x = 0; x < NE; ++x) acc[k][x] = 0.f;
        for (int p = 0; p < n; p += 64) {
            const uint64_t wcur = wnext;
            const int m = n - p < 64 ? n - p : 64;  // lookups in this window
            const int wlo = (int)(uint32_t)wcur, whi = (int)(uint32_t)(wcur >> 32);
            // one sub-block of U load instructions; FULL: all UR lookups are
            // in the bag (no masking).  The two forms are separate code paths
            // so that no loaded value has to be merged (and waited for) early.
            auto sub_block = [&](int s, auto full_tag) {
                constexpr bool FULL = decltype(full_tag)::value;
                V v[U];
                const int bidx = (s + h) * 4;  // bpermute byte index of lookup s + h
                if constexpr (FULL) {
                    uint32_t lo[U], hi[U];
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        lo[u] = (uint32_t)__builtin_amdgcn_ds_bpermute(bidx + u * R * 4, wlo);
                        hi[u] = (uint32_t)__builtin_amdgcn_ds_bpermute(bidx + u * R * 4, whi);
                    }
#pragma unroll
                    for (int u = 0; u < U; ++u) v[u] = wload<V>(((uint64_t)hi[u] << 32) | lo[u], eoff);
                } else {
#pragma unroll
                    for (int u = 0; u < U; ++u)
                        if (s + u * R < m) {
                            const uint32_t lo = (uint32_t)__builtin_amdgcn_ds_bpermute(bidx + u * R * 4, wlo);
                            const uint32_t hi = (uint32_t)__builtin_amdgcn_ds_bpermute(bidx + u * R * 4, whi);
                            if (s + u * R + h < m) v[u] = wload<V>(((uint64_t)hi << 32) | lo, eoff);
                        }
                }
                if (s == 0) {
                    // the next window, issued after this sub-block's row loads
                    asm volatile("" ::: "memory");
                    if (p + 64 < n) wnext = RECMG_GLOBAL(uint64_t, raddr + a + p + 64 + lane);
                    else next_bag_window(b);
                }
#pragma unroll
                for (int u = 0; u < U; ++u)
                    if (FULL || s + u * R + h < m) wadd<DT, LW>(acc[u % NA], v[u]);
            };
            int s = 0;
            for (; s + UR <= m; s += UR) sub_block(s, std::true_type{});
            if (s < m) sub_block(s, std::false_type{});
        }
        wstore<NE, R, NA>(acc, h, obase + (int64_t)b * D + gl * NE);
    }
}

#ifndef RECMG_WPOOL_OCC
#define RECMG_WPOOL_OCC 1
#endif

// RECMG_WPOOL_OCC: waves per SIMD the register allocation must allow
// nbt > 0: every table of the launch has nbt blocks, so block lb belongs to
// table btab[k0 + (lb - boff) / nbt] (no search; one wave's prologue is a
// chain of dependent loads, and the search would add four to it).
template <int DT, int LW, int R>
__global__ void __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(RECMG_WPOOL_OCC))) k_pool_w(DGlobal g, const int64_t *__restrict__ offsets,
                                                   const uint64_t *__restrict__ raddr, int32_t B,
                                                   float *__restrict__ out, const int32_t *__restrict__ bstart,
                                                   const int32_t *__restrict__ btab, int32_t nt, int32_t boff,
                                                   int32_t nblk, int32_t k0, int32_t nbt) {
    const int lb = boff + xcd_block(nblk);
    int k, b0;
    if (nbt > 0) {
        k = k0 + (lb - boff) / nbt;
        b0 = boff + (k - k0) * nbt;
    } else {
        k = find_seg32(bstart, nt, lb);
        b0 = bstart[k];
    }
    const int t = btab[k];
    const int err = *g.err;
    const DTable &tb = g.tabs[t];
    const int D = tb.dim;
    const int64_t ooff = (int64_t)B * tb.out_elem_off;
    if (err) return;
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
    const int j0 = ((lb - b0) * (kBlock / 64) + wave) * kWaveBags;
    if (j0 >= B) return;
    const int nbags = B - j0 < kWaveBags ? B - j0 : kWaveBags;
    const int64_t *ob = offsets + (int64_t)t * B + j0;
    float *ob_out = out + ooff + (int64_t)j0 * D;
    if constexpr (R == 1) pool_wave_s<DT, LW>(raddr, ob, nbags, tb.wnch, D, ob_out);
    else pool_wave_v<DT, LW, R>(raddr, ob, nbags, D, ob_out);
}

// Publishes the forward's counters; log_slot >= 0: also as that call's record
// of the stats log (the placement group of the record stays zero).
__global__ void k_fwd_finalize(DGlobal g, int64_t log_slot) {
    if (*g.err) return;
    for (int t = threadIdx.x; t < g.T; t += blockDim.x) {
        TState &st = g.st[t];
        const DTable &tb = g.tabs[t];
        int64_t v[kFwdStats];
        v[0] = g.tstart[t + 1] - g.tstart[t];
        v[1] = st.ucount;
        v[2] = st.hits;
        v[3] = st.hits_pf;
        v[4] = st.mcount;
        v[5] = (int64_t)st.mcount * tb.row_bytes;
        v[6] = st.covered;
        for (int k = 0; k < kFwdStats; ++k) {
            st.last[k] = v[k];
            st.total[k] += v[k];
        }
        if (log_slot >= 0) {
            int64_t *rec = g.stat_log + (log_slot * g.T + t) * (kNumStats + 1);
            for (int k = 0; k <= kNumStats; ++k) rec[k] = k < kFwdStats ? v[k] : 0;
        }
    }
}

// ----------------------------------------------------------------- launchers

static inline unsigned grid_for(int64_t n, int per_block, unsigned cap) {
    int64_t b = (n + per_block - 1) / per_block;
    if (b < 1) b = 1;
    if (b > (int64_t)cap) b = cap;
    return (unsigned)b;
}

void launch_fwd_prep(const DGlobal &g, const int64_t *offsets, int32_t B, int64_t n, hipStream_t s) {
    const int64_t items = ((int64_t)g.T * B + 1) > (g.T + 1) ? ((int64_t)g.T * B + 1) : (g.T + 1);
    k_fwd_prep<<<(unsigned)((items + kBlock - 1) / kBlock), kBlock, 0, s>>>(g, offsets, B, n);
}

void launch_fwd_probe(const DGlobal &g, int32_t stamp, int64_t n, hipStream_t s) {
    if (n <= 0) return;
    k_fwd_probe<<<grid_for(n, kBlock, 8192), kBlock, 0, s>>>(g, stamp, n);
}

void launch_fwd_cover(const DGlobal &g, int32_t stamp, int64_t np, hipStream_t s) {
    if (np <= 0) return;
    k_fwd_cover<<<grid_for(np, kBlock, 4096), kBlock, 0, s>>>(g, stamp, np);
}

void launch_fwd_src(const DGlobal &g, const int32_t *indices, int64_t n, hipStream_t s) {
    if (n <= 0) return;
    k_fwd_src<<<grid_for(n, kBlock * items_per_thread(n, 4), 16384), kBlock, 0, s>>>(g, indices, n);
}

#ifndef RECMG_FETCH_BLOCKS
#define RECMG_FETCH_BLOCKS 96
#endif

// As for the prefetch fill, which runs at the same time on the copy stream: a
// modest grid fills the host link and leaves most CUs' L1s to other kernels
// (the next placement runs beside it).  Measured on configuration 3 (64-256
// blocks): 96 is best with 32-way sets (k_sa_place's critical path runs
// alongside), within 1% of the best without prefetch and on configuration 5.
void launch_fetch(const DGlobal &g, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    if (ev0 || ev1) hipExtLaunchKernelGGL(k_fetch, dim3(RECMG_FETCH_BLOCKS), dim3(kBlock), 0, s, ev0, ev1, 0, g);
    else k_fetch<<<RECMG_FETCH_BLOCKS, kBlock, 0, s>>>(g);
}

int pool_kind(int dtype, int vec, int wlw, int wr) {
    if (wlw == 0) return dtype * 2 + vec;
    const int v = wlw == 16 ? (wr == 1 ? 0 : wr == 2 ? 1 : 2) : wlw == 8 ? 3 : 4;
    return kPoolKindsGroup + dtype * 5 + v;
}

// ev0 / ev1 (may be null): recorded by the first / last dispatch itself, so
// they bracket the kernels' execution without the dispatch gap.
void launch_pool(const DGlobal &g, const int64_t *offsets, int32_t B, float *out, const int32_t *bstart,
                 const int32_t *btab, int32_t nt, const PoolLaunch *ls, int nl, hipEvent_t ev0, hipEvent_t ev1,
                 hipStream_t s) {
    using KG = void (*)(DGlobal, const int64_t *, int32_t, float *, const int32_t *, const int32_t *, int32_t,
                        int32_t, int32_t);
    using KW = void (*)(DGlobal, const int64_t *, const uint64_t *, int32_t, float *, const int32_t *,
                        const int32_t *, int32_t, int32_t, int32_t, int32_t, int32_t);
    static const KG kg[kPoolKindsGroup] = {k_pool<RECMG_F32, false>,  k_pool<RECMG_F32, true>,
                                           k_pool<RECMG_F16, false>,  k_pool<RECMG_F16, true>,
                                           k_pool<RECMG_BF16, false>, k_pool<RECMG_BF16, true>};
#define RECMG_WK(DT) k_pool_w<DT, 16, 1>, k_pool_w<DT, 16, 2>, k_pool_w<DT, 16, 4>, k_pool_w<DT, 8, 4>, k_pool_w<DT, 4, 4>
    static const KW kw[kPoolKinds - kPoolKindsGroup] = {RECMG_WK(RECMG_F32), RECMG_WK(RECMG_F16),
                                                        RECMG_WK(RECMG_BF16)};
#undef RECMG_WK
    int first = -1, last = -1;
    for (int i = 0; i < nl; ++i)
        if (ls[i].nblk > 0) {
            if (first < 0) first = i;
            last = i;
        }
    for (int i = 0; i < nl; ++i) {
        const PoolLaunch &L = ls[i];
        if (L.nblk <= 0) continue;
        hipEvent_t a = i == first ? ev0 : nullptr, b = i == last ? ev1 : nullptr;
        const dim3 grid((unsigned)L.nblk), blk(kBlock);
        if (L.kind < kPoolKindsGroup) {
            const KG k = kg[L.kind];
            if (a || b) hipExtLaunchKernelGGL(k, grid, blk, 0, s, a, b, 0, g, offsets, B, out, bstart, btab, nt,
                                              L.boff, L.nblk);
            else k<<<grid, blk, 0, s>>>(g, offsets, B, out, bstart, btab, nt, L.boff, L.nblk);
        } else {
            const KW k = kw[L.kind - kPoolKindsGroup];
            const uint64_t *ra = g.raddr;
            if (a || b) hipExtLaunchKernelGGL(k, grid, blk, 0, s, a, b, 0, g, offsets, ra, B, out, bstart, btab, nt,
                                              L.boff, L.nblk, L.k0, L.nbt);
            else k<<<grid, blk, 0, s>>>(g, offsets, ra, B, out, bstart, btab, nt, L.boff, L.nblk, L.k0, L.nbt);
        }
    }
}

void launch_fwd_finalize(const DGlobal &g, int64_t log_slot, hipStream_t s) {
    k_fwd_finalize<<<1, kBlock, 0, s>>>(g, log_slot);
}

}  // namespace recmg
