// Device-side pieces shared by the solver kernels: the per-instance state
// view, flow-list lookups, the predecessor walk, and small wave/block utils.
#pragma once

#include "mcf_internal.h"

namespace gwtf {
namespace dev {

constexpr int kPredSplit = -1; // entry: from own exit (reverse compute); exit: from own entry
constexpr int kPredSrc = -2;   // entry of stage 0: from the data node
constexpr int kPredNone = -3;
constexpr int kStatusInternal = 3; // solver self-check failed (never expected)

template <bool NARROW> struct Types;
template <> struct Types<true> {
    using pred = int8_t;
    using off = uint16_t;
    using len = uint8_t;
    using part = uint8_t;
};
template <> struct Types<false> {
    using pred = int16_t;
    using off = int32_t;
    using len = uint16_t;
    using part = uint16_t;
};

template <bool NARROW> struct State {
    using T = Types<NARROW>;
    int32_t *din, *dout, *pout, *flow, *cap, *cost, *srcc, *snkc;
    uint64_t *pend;
    typename T::pred *prin, *prout;
    typename T::off *loff;
    typename T::len *llen;
    int32_t *lcost, *lamt;
    typename T::part *lpart;

    __device__ void carve(unsigned char *base, const StateLayout &L)
    {
        din = reinterpret_cast<int32_t *>(base + L.din);
        dout = reinterpret_cast<int32_t *>(base + L.dout);
        pout = reinterpret_cast<int32_t *>(base + L.pout);
        flow = reinterpret_cast<int32_t *>(base + L.flow);
        cap = reinterpret_cast<int32_t *>(base + L.cap);
        cost = reinterpret_cast<int32_t *>(base + L.cost);
        pend = reinterpret_cast<uint64_t *>(base + L.pend);
        srcc = reinterpret_cast<int32_t *>(base + L.srcc);
        snkc = reinterpret_cast<int32_t *>(base + L.snkc);
        prin = reinterpret_cast<typename T::pred *>(base + L.prin);
        prout = reinterpret_cast<typename T::pred *>(base + L.prout);
        loff = reinterpret_cast<typename T::off *>(base + L.loff);
        llen = reinterpret_cast<typename T::len *>(base + L.llen);
        lcost = reinterpret_cast<int32_t *>(base + L.lcost);
        lamt = reinterpret_cast<int32_t *>(base + L.lamt);
        lpart = reinterpret_cast<typename T::part *>(base + L.lpart);
    }
};

struct Shared {
    long long F, cost;
    long long rows, pulls, rounds, augs;
    unsigned long long tbest;
    int Dt, predt, pit, any, bad, maxc, status, route;
    long long slots;
};

__device__ __forceinline__ uint64_t lap(uint64_t &tick)
{
    uint64_t now = wall_clock64(), d = now - tick;
    tick = now;
    return d;
}

// Reduction over the 64 lanes with DPP moves only (no LDS): swaps within
// quads, rotations within rows of 16, then row broadcasts; lane 63 ends with
// the result, which every lane reads.
template <int kCtrl, int kRows> __device__ __forceinline__ uint32_t dpp_mov(uint32_t x)
{
    return uint32_t(__builtin_amdgcn_update_dpp(int(x), int(x), kCtrl, kRows, 0xf, false));
}
template <bool kMax> __device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t v)
{
    auto op = [](uint32_t a, uint32_t b) { return kMax ? max(a, b) : min(a, b); };
    v = op(v, dpp_mov<0xb1, 0xf>(v));  // quad_perm [1,0,3,2]
    v = op(v, dpp_mov<0x4e, 0xf>(v));  // quad_perm [2,3,0,1]
    v = op(v, dpp_mov<0x124, 0xf>(v)); // row_ror:4
    v = op(v, dpp_mov<0x128, 0xf>(v)); // row_ror:8
    v = op(v, dpp_mov<0x142, 0xa>(v)); // row_bcast:15 into rows 1 and 3
    v = op(v, dpp_mov<0x143, 0xc>(v)); // row_bcast:31 into rows 2 and 3
    return __builtin_amdgcn_readlane(v, 63);
}

__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Bits b of a 64-bit word (row i = 64*word + b) with i % WAVES == w.
template <int WAVES> __device__ __forceinline__ uint64_t wave_rows(int w)
{
    uint64_t m = 0;
#pragma unroll
    for (int b = 0; b < 64; b += WAVES) m |= uint64_t(1) << b;
    return m << w;
}

template <int NT> __device__ int block_exclusive_scan(int v, int *buf, int &total)
{
    const int tid = threadIdx.x;
    buf[tid] = v;
    __syncthreads();
    for (int d = 1; d < NT; d <<= 1) {
        int add = tid >= d ? buf[tid - d] : 0;
        __syncthreads();
        buf[tid] += add;
        __syncthreads();
    }
    total = buf[NT - 1];
    int excl = buf[tid] - v;
    __syncthreads();
    return excl;
}

template <bool NARROW>
__device__ int list_find(const State<NARROW> &st, int q, int j)
{
    int off = st.loff[q], len = st.llen[q];
    for (int e = off; e < off + len; ++e)
        if (st.lpart[e] == j) return e;
    return -1;
}

// Walks the predecessor chain from the sink.  APPLY = false returns the
// bottleneck residual; APPLY = true pushes delta along the chain.  A link
// leaving exit(k,i) is applied together with the reverse link that enters
// exit(k,i) (if any), decrement first, so a flow list never holds more
// partners than its capacity.
// Returns -1 if the chain is inconsistent (longer than the vertex count or
// naming a link missing from a flow list): a solver fault, reported as an
// internal-error status rather than followed.
template <bool APPLY, bool NARROW>
__device__ int walk_path(State<NARROW> &st, const int32_t *gac, int S, int n, int supply, int predt,
                         int delta)
{
    int k = S - 1, i = predt;
    bool at_exit = true;
    if (predt < 0 || predt >= n) return -1;
    for (int steps = 0;; ++steps) {
        if (steps > 2 * S * n + 4) return -1;
        if (at_exit) {
            int q = k * n + i;
            int pr = st.prout[q];
            if (pr == kPredSplit) {
                if (APPLY) st.flow[q] += delta;
                else delta = min(delta, st.cap[q] - st.flow[q]);
                at_exit = false;
            } else {
                if (pr < 0 || k + 1 >= S) return -1;
                int e = list_find(st, q, pr);
                if (e < 0) return -1;
                if (APPLY) {
                    int left = st.lamt[e] - delta;
                    if (left == 0) {
                        int last = st.loff[q] + st.llen[q] - 1;
                        st.lpart[e] = st.lpart[last];
                        st.lamt[e] = st.lamt[last];
                        st.lcost[e] = st.lcost[last];
                        st.llen[q] = st.llen[q] - 1;
                    } else {
                        st.lamt[e] = left;
                    }
                } else {
                    delta = min(delta, st.lamt[e]);
                }
                k = k + 1;
                i = pr;
                at_exit = false;
            }
        } else {
            int q = k * n + i;
            int pr = st.prin[q];
            if (pr == kPredSrc) break;
            if (pr == kPredSplit) {
                if (APPLY) st.flow[q] -= delta;
                else delta = min(delta, st.flow[q]);
                at_exit = true;
            } else {
                // forward link exit(k-1, pr) -> entry(k, i): unbounded residual
                if (pr < 0 || k < 1) return -1;
                int q2 = (k - 1) * n + pr;
                if (APPLY) {
                    int pr2 = st.prout[q2];
                    if (pr2 != kPredSplit) {
                        // reverse link entry(k, pr2) -> exit(k-1, pr) comes first
                        int e = list_find(st, q2, pr2);
                        if (e < 0) return -1;
                        int left = st.lamt[e] - delta;
                        if (left == 0) {
                            int last = st.loff[q2] + st.llen[q2] - 1;
                            st.lpart[e] = st.lpart[last];
                            st.lamt[e] = st.lamt[last];
                            st.lcost[e] = st.lcost[last];
                            st.llen[q2] = st.llen[q2] - 1;
                        } else {
                            st.lamt[e] = left;
                        }
                    }
                    int e = list_find(st, q2, i);
                    if (e >= 0) {
                        st.lamt[e] += delta;
                    } else {
                        if (st.llen[q2] >= min(min(st.cap[q2], n), supply)) return -1;
                        int at = st.loff[q2] + st.llen[q2];
                        st.lpart[at] = i;
                        st.lamt[at] = delta;
                        st.lcost[at] = gac[size_t(q2) * n + i];
                        st.llen[q2] = st.llen[q2] + 1;
                    }
                    if (pr2 != kPredSplit) {
                        // continue at entry(k, pr2): exit(k-1, pr) is done
                        i = pr2;
                        at_exit = false;
                        continue;
                    }
                    st.flow[q2] += delta; // compute arc entry(k-1,pr) -> exit(k-1,pr)
                    k = k - 1;
                    i = pr;
                    at_exit = false;
                    continue;
                }
                k = k - 1;
                i = pr;
                at_exit = true;
            }
        }
    }
    return delta;
}

} // namespace dev
} // namespace gwtf
