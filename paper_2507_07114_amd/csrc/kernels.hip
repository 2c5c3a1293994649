// HIP kernels of the lossy step for gfx950 and their launchers.
//
// Work decomposition shared by every per-packet kernel: a workgroup owns a
// chunk of one packet covering 4 KiB of each row it streams (256 threads =
// 4 wave64s and 2048 elements for bf16 rows, 128 threads and 1024 elements
// for fp32 rows); thread t owns elements [8t, 8t + 8) of the chunk, so each
// row read or written is one 16-byte (bf16) or two 16-byte (fp32) accesses
// per thread and a wavefront touches 1 KiB (bf16) or 2 KiB (fp32) of
// contiguous HBM.
// The masks of the packet sit in LDS as 64-bit words; loops over arrived or
// stale rows walk the set bits with scalar (wave-uniform) control flow, so
// a lost packet costs no memory traffic and causes no divergence.
#include "kernels.h"

#include <math.h>

#include <atomic>
#include <mutex>

namespace lossy {

// ---------------------------------------------------------------------------
// Masks
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void k_masks_bernoulli(int n, int64_t num_packets,
                                                              uint64_t step, uint64_t dir,
                                                              uint64_t seed, uint64_t thr,
                                                              int owner, const uint8_t* reliable,
                                                              uint8_t* arrived) {
    const int64_t total = (int64_t)n * num_packets;
    for (int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * kThreads) {
        const int64_t i = idx / num_packets;
        const int64_t k = idx - i * num_packets;
        const bool a = bernoulli_arrived((uint64_t)k, (uint64_t)i, step, dir, seed, thr) ||
                       forced_arrival((int)i, k, owner, reliable);
        arrived[idx] = a ? 1 : 0;
    }
}

// Bernoulli masks of one or two directions in one launch (job j covers
// entries [j n P, (j + 1) n P) of the grid).
struct MaskJobs {
    MaskJob job[2];
};

__global__ __launch_bounds__(kThreads) void k_masks_bernoulli_jobs(int n, int64_t num_packets,
                                                                   uint64_t step, int njobs,
                                                                   MaskJobs J) {
    const int64_t per = (int64_t)n * num_packets;
    const int64_t total = per * njobs;
    for (int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * kThreads) {
        const int j = idx >= per ? 1 : 0;
        const MaskJob& m = J.job[j];
        const int64_t e = idx - j * per;
        const int64_t i = e / num_packets;
        const int64_t k = e - i * num_packets;
        const bool a = bernoulli_arrived((uint64_t)k, (uint64_t)i, step, m.dir, m.seed, m.thr) ||
                       forced_arrival((int)i, k, m.owner, m.reliable);
        m.arrived[e] = a ? 1 : 0;
    }
}

// Bernoulli masks with parity packets.  A workgroup takes `span` consecutive
// packets of one (direction, row), one packet per thread, span a multiple of
// G.  Each thread draws its packet's arrival and applies the transfers that
// cannot be lost, and the first span / G threads draw the arrival of one
// group's parity packet each (counter (group, row, step, dir + 2)); ballots
// put both bitmaps in LDS.  A lost packet whose group (G consecutive packets)
// lost nothing else is rebuilt when the group's parity packet arrived: XOR
// of the parity with the other G - 1 packets gives it back exactly.
__global__ __launch_bounds__(kThreads) void k_masks_parity(ParityLaunch L) {
    __shared__ uint64_t s_lost[kThreads / 64];
    __shared__ uint64_t s_par[kThreads / 64];
    const int64_t per_dir = (int64_t)L.n * L.spans;
    const int64_t b = blockIdx.x;
    const int s = b >= per_dir ? 1 : 0;
    const MaskJob& J = L.job[s];
    const int64_t rem = b - s * per_dir;
    const int64_t i = rem / L.spans;
    const int64_t k0 = (rem - i * L.spans) * L.span;
    const int t = threadIdx.x;
    const int64_t k = k0 + t;
    const bool in = t < L.span && k < L.P;
    bool a = true;
    if (in)
        a = bernoulli_arrived((uint64_t)k, (uint64_t)i, L.step, J.dir, J.seed, J.thr) ||
            forced_arrival((int)i, k, J.owner, J.reliable);
    // thread t < span / G: parity packet of group k0 / G + t (if the group exists)
    bool par = false;
    if (t < L.span / L.G && k0 + (int64_t)t * L.G < L.P)
        par = bernoulli_arrived((uint64_t)(k0 / L.G + t), (uint64_t)i, L.step, J.dir + 2, J.seed,
                                J.thr);
    const uint64_t lost = __ballot(!a);
    const uint64_t pbits = __ballot(par);
    if ((t & 63) == 0) {
        s_lost[t >> 6] = lost;
        s_par[t >> 6] = pbits;
    }
    __syncthreads();
    if (!in) return;
    if (!a) {
        const int gl = t / L.G;                                // group within the span
        const int g0 = gl * L.G;                               // its first thread
        const int g1 = g0 + L.G < L.span ? g0 + L.G : L.span;  // one past its last
        int missing = 0;
        for (int w = g0 >> 6; w <= (g1 - 1) >> 6; ++w) {
            const int lo = g0 > w * 64 ? g0 - w * 64 : 0;
            const int hi = g1 < (w + 1) * 64 ? g1 - w * 64 : 64;
            const uint64_t keep = (hi == 64 ? ~0ull : ((1ull << hi) - 1)) & ~((1ull << lo) - 1);
            missing += __popcll(s_lost[w] & keep);
        }
        if (missing == 1) a = (s_par[gl >> 6] >> (gl & 63)) & 1;
    }
    J.arrived[i * L.P + k] = a ? 1 : 0;
}

// Gilbert-Elliott masks.  A chain's per-packet transition is a map on
// {Good, Bad}, encoded in two bits (bit 0 = image of Good, bit 1 = image of
// Bad); maps compose associatively, so the chain state before any packet is
// a prefix composition.  Two launches over (direction, worker, segment of
// kGeSeg packets) workgroups:
//   compose: each thread composes the maps of its run of kGeRun packets and
//            stores the composite; a block scan gives the segment composite.
//   apply:   each workgroup folds the composites of the earlier segments of
//            its chain into its start state, scans its threads' composites
//            for each run's start state, and replays its runs, emitting
//            arrivals; the last run of the last segment stores the end state.
// The input state is copied aside by the first launch so that the second can
// overwrite the caller's state without racing its own readers.
constexpr uint32_t kGeIdentity = 0x2u;  // Good -> Good, Bad -> Bad

__device__ __forceinline__ uint32_t ge_apply(uint32_t map, uint32_t s) { return (map >> s) & 1u; }

// (g after f)
__device__ __forceinline__ uint32_t ge_compose(uint32_t g, uint32_t f) {
    return ge_apply(g, ge_apply(f, 0)) | (ge_apply(g, ge_apply(f, 1)) << 1);
}

__device__ __forceinline__ uint32_t ge_packet_map(uint64_t u0, const GeParams& ge) {
    return (u0 < ge.thr_gb ? 1u : 0u) | ((u0 < ge.thr_bg ? 0u : 1u) << 1);
}

// In-place inclusive scan of kThreads maps: s[t] = f_t o ... o f_0.
__device__ __forceinline__ void ge_block_scan(uint32_t* s) {
    for (int off = 1; off < kThreads; off <<= 1) {
        const uint32_t mine = s[threadIdx.x];
        const uint32_t before = (int)threadIdx.x >= off ? s[threadIdx.x - off] : kGeIdentity;
        __syncthreads();
        s[threadIdx.x] = ge_compose(mine, before);
        __syncthreads();
    }
}

struct GeBlock {
    int dir, i;
    int64_t s;
    int64_t k0, k1;  // this thread's run
};

__device__ __forceinline__ GeBlock ge_block(const GeLaunch& L) {
    GeBlock b;
    const int64_t per_dir = (int64_t)L.n * L.S;
    const int64_t id = blockIdx.x;
    b.dir = (int)(id / per_dir);
    const int64_t rem = id - b.dir * per_dir;
    b.i = (int)(rem / L.S);
    b.s = rem - (int64_t)b.i * L.S;
    b.k0 = b.s * kGeSeg + (int64_t)threadIdx.x * kGeRun;
    b.k1 = b.k0 + kGeRun < L.P ? b.k0 + kGeRun : L.P;
    return b;
}

__global__ __launch_bounds__(kThreads) void k_ge_compose(GeLaunch L) {
    __shared__ uint32_t s_map[kThreads];
    const GeBlock b = ge_block(L);
    const GeJob& J = L.job[b.dir];
    uint32_t f = kGeIdentity;
    for (int64_t k = b.k0; k < b.k1; ++k) {
        uint64_t w0, w1;
        philox4x64_10((uint64_t)k, (uint64_t)b.i, L.step, J.dir, J.ge.seed, 0, w0, w1);
        f = ge_compose(ge_packet_map(w0 >> 32, J.ge), f);
    }
    const int64_t seg = (int64_t)b.i * L.S + b.s;
    J.tmaps[seg * kThreads + threadIdx.x] = (uint8_t)f;
    s_map[threadIdx.x] = f;
    __syncthreads();
    ge_block_scan(s_map);
    if (threadIdx.x == kThreads - 1) J.comps[seg] = (uint8_t)s_map[kThreads - 1];
    if (b.s == 0 && threadIdx.x == 0) J.state_in[b.i] = J.state[b.i] ? 1 : 0;
}

__global__ __launch_bounds__(kThreads) void k_ge_apply(GeLaunch L) {
    __shared__ uint32_t s_run[kThreads];
    __shared__ uint32_t s_seg[kThreads];
    const GeBlock b = ge_block(L);
    const GeJob& J = L.job[b.dir];
    const int64_t row = (int64_t)b.i * L.S;
    // Composition of the earlier segments of this chain, 256 at a time.
    uint32_t before = kGeIdentity;
    for (int64_t base = 0; base < b.s; base += kThreads) {
        const int64_t j = base + threadIdx.x;
        s_seg[threadIdx.x] = j < b.s ? J.comps[row + j] : kGeIdentity;
        __syncthreads();
        ge_block_scan(s_seg);
        before = ge_compose(s_seg[kThreads - 1], before);
        __syncthreads();
    }
    s_run[threadIdx.x] = J.tmaps[(row + b.s) * kThreads + threadIdx.x];
    __syncthreads();
    ge_block_scan(s_run);
    const uint32_t own_prefix = threadIdx.x == 0 ? kGeIdentity : s_run[threadIdx.x - 1];
    uint32_t x = ge_apply(own_prefix, ge_apply(before, J.state_in[b.i]));
    for (int64_t k = b.k0; k < b.k1; ++k) {
        uint64_t w0, w1;
        philox4x64_10((uint64_t)k, (uint64_t)b.i, L.step, J.dir, J.ge.seed, 0, w0, w1);
        x = ge_apply(ge_packet_map(w0 >> 32, J.ge), x);
        const bool lost = (w1 >> 32) < (x ? J.ge.thr_loss_bad : J.ge.thr_loss_good);
        const bool a = !lost || forced_arrival(b.i, k, J.owner, J.reliable);
        J.arrived[(int64_t)b.i * L.P + k] = a ? 1 : 0;
    }
    if (b.s == L.S - 1 && threadIdx.x == kThreads - 1) J.state[b.i] = (uint8_t)x;
}

template <int NT>
__device__ __forceinline__ Chunk chunk_of(int64_t d, int64_t L, int cpp) {
    return chunk_at<NT>(blockIdx.x, d, L, cpp);
}

// ---------------------------------------------------------------------------
// One-stage entry points
// ---------------------------------------------------------------------------
template <class G, bool W>
__device__ __forceinline__ void aggregate_chunk(const AggParams& p, const Chunk& ch,
                                                const uint64_t* words, int K) {
    float th[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (K == 0 && p.lam != 0.0f && p.var.kind == kEstArrivedMean)
        load8<F32, W>(p.theta + ch.e0, ch.nv, th);
    const bool relp = p.var.reliable != nullptr && p.var.reliable[ch.k] != 0;
    float g[8];
    aggregate8<G, W>(reinterpret_cast<const typename G::T*>(p.grads), p.ld, ch, words, p.n, K,
                     p.lam, th, p.var, relp, NoPace(), g);
    store_f32x8<W>(p.g_hat + ch.e0, ch.nv, g);
}

template <class G>
__global__ __launch_bounds__(G::kPacketThreads) void k_aggregate(AggParams p) {
    constexpr int NT = G::kPacketThreads;
    __shared__ uint64_t s_words[1][kMaxWords];
    const Chunk ch = chunk_of<NT>(p.d, p.L, p.cpp);
    const MaskSource src[1] = {{false, 0, 0, p.arrived, -1, nullptr}};
    const int dirs[1] = {0};
    stage_masks<NT, 1>(src, p.n, p.P, ch.k, 0, dirs, s_words);
    const int nw = (p.n + 63) >> 6;
    const int K = popcount_words(s_words[0], nw);
    if (ch.c == 0 && threadIdx.x == 0 && p.counts) p.counts[ch.k] = K;
    if (ch.nv == 0) return;
    if (ch.whole) aggregate_chunk<G, true>(p, ch, s_words[0], K);
    else aggregate_chunk<G, false>(p, ch, s_words[0], K);
}

template <bool W>
__device__ __forceinline__ void shard_step8(int64_t e0, int nv, const OptParams& o, float* theta,
                                            float* m, float* v, const float* g_hat) {
    float th[8], mm[8], vv[8], g[8];
    load8<F32, W>(theta + e0, nv, th);
    load8<F32, W>(g_hat + e0, nv, g);
    if (o.kind >= 1) load8<F32, W>(m + e0, nv, mm);
    if (o.kind == 2) load8<F32, W>(v + e0, nv, vv);
    update8(o, th, mm, vv, g);
    store_f32x8<W>(theta + e0, nv, th);
    if (o.kind >= 1) store_f32x8<W>(m + e0, nv, mm);
    if (o.kind == 2) store_f32x8<W>(v + e0, nv, vv);
}

__global__ __launch_bounds__(kThreads) void k_shard_step(int64_t d, OptParams o, float* theta,
                                                         float* m, float* v,
                                                         const float* g_hat) {
    const int64_t b0 = (int64_t)blockIdx.x * kThreads * kElems;
    const int64_t e0 = b0 + (int64_t)threadIdx.x * kElems;
    if (e0 >= d) return;
    const int nv = d - e0 >= 8 ? 8 : (int)(d - e0);
    if (d % 8 == 0 || d >= b0 + kThreads * kElems) shard_step8<true>(e0, nv, o, theta, m, v, g_hat);
    else shard_step8<false>(e0, nv, o, theta, m, v, g_hat);
}

template <class R, bool W>
__device__ __forceinline__ void broadcast_chunk(const BcastParams& p, const Chunk& ch,
                                                const uint64_t* words, int nw) {
    float th[8];
    load8<F32, W>(p.theta + ch.e0, ch.nv, th);
    Packed8<R> r;
    r.pack(th);
    typename R::T* reps = reinterpret_cast<typename R::T*>(p.replicas);
    for (int w = 0; w < nw; ++w) {
        uint64_t bits = uniform64(words[w]);
        while (bits) {
            const int i = w * 64 + __builtin_ctzll(bits);
            bits &= bits - 1;
            r.template store<W>(reps + (int64_t)i * p.ld + ch.e0, ch.nv);
        }
    }
}

template <class R>
__global__ __launch_bounds__(R::kPacketThreads) void k_broadcast(BcastParams p) {
    constexpr int NT = R::kPacketThreads;
    __shared__ uint64_t s_words[1][kMaxWords];
    const Chunk ch = chunk_of<NT>(p.d, p.L, p.cpp);
    const MaskSource src[1] = {{false, 0, 0, p.arrived, -1, nullptr}};
    const int dirs[1] = {1};
    stage_masks<NT, 1>(src, p.n, p.P, ch.k, 0, dirs, s_words);
    if (ch.nv == 0) return;
    const int nw = (p.n + 63) >> 6;
    if (ch.whole) broadcast_chunk<R, true>(p, ch, s_words[0], nw);
    else broadcast_chunk<R, false>(p, ch, s_words[0], nw);
}

// Drift of one chunk over all rows, read in ascending order.
template <class R, bool W>
__device__ __forceinline__ void drift_chunk(const DriftParams& p, const Chunk& ch, double& pair,
                                            double& range, double& abs_sum) {
    const typename R::T* reps = reinterpret_cast<const typename R::T*>(p.replicas);
    float r[8];
    if (p.theta) {
        float th[8];
        load8<F32, W>(p.theta + ch.e0, ch.nv, th);
        Packed8<R> pr;
        pr.pack(th);
#pragma unroll
        for (int j = 0; j < 8; ++j) r[j] = pr.value(j);
    } else {
        load8<R, W>(reps + ch.e0, ch.nv, r);
    }
    Drift8<FloatBounds8> acc;
    acc.init(false, r);
    for (int i0 = 0; i0 < p.n; i0 += kBatchDrift) {
        Raw8<R> raw[kBatchDrift];
#pragma unroll
        for (int u = 0; u < kBatchDrift; ++u) {
            const int row = i0 + u < p.n ? i0 + u : i0;
            load_raw<W>(reps + (int64_t)row * p.ld + ch.e0, ch.nv, raw[u]);
        }
#pragma unroll
        for (int u = 0; u < kBatchDrift; ++u) {
            if (i0 + u < p.n) {
                float x[8];
                unpack(raw[u], x);
                acc.add(x, r, ch.nv);
            }
        }
    }
    acc.finish(p.n, ch.nv, pair, range);
    abs_sum = acc.abs_sum;
}

template <class R>
__global__ __launch_bounds__(R::kPacketThreads) void k_drift(DriftParams p) {
    constexpr int NT = R::kPacketThreads;
    __shared__ uint64_t s_words[1][kMaxWords];
    const Chunk ch = chunk_of<NT>(p.d, p.L, p.cpp);
    const int nw = (p.n + 63) >> 6;
    uint32_t stale = 0;
    if (p.arrived) {
        const MaskSource src[1] = {{false, 0, 0, p.arrived, -1, nullptr}};
        const int dirs[1] = {1};
        stage_masks<NT, 1>(src, p.n, p.P, ch.k, 0, dirs, s_words);
        if (ch.c == 0) stale = (uint32_t)(p.n - popcount_words(s_words[0], nw));
    }
    double pair = 0.0, range = 0.0, abs_sum = 0.0;
    if (ch.nv > 0) {
        if (ch.whole) drift_chunk<R, true>(p, ch, pair, range, abs_sum);
        else drift_chunk<R, false>(p, ch, pair, range, abs_sum);
    }
    block_reduce_partial<NT>(pair, abs_sum, range, stale, 0, p.partials + blockIdx.x);
    if (blockIdx.x == 0 && threadIdx.x == 0) *reduce_counter(p.groups) = 0u;
}

// Fixed-order reduction of the per-workgroup partials into the ll_drift
// record.
// Fixed-order tree over the workgroup; thread 0 returns the total.
template <int NT>
__device__ __forceinline__ DriftAcc block_fold(DriftAcc a) {
    __shared__ DriftAcc s_acc[NT];
    s_acc[threadIdx.x] = a;
    __syncthreads();
    for (int off = NT / 2; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) s_acc[threadIdx.x].add(s_acc[threadIdx.x + off]);
        __syncthreads();
    }
    return s_acc[0];
}

// Counts one finished workgroup once this thread's earlier stores have
// completed.  The group totals are written with device-coherent stores and
// read with device-coherent loads, so waiting for the stores is all the
// ordering needed (a device-scope fence would also write back the L2).
__device__ __forceinline__ unsigned count_done(unsigned* counter) {
    __builtin_amdgcn_s_waitcnt(0);
    return __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The ll_drift record from the folded totals (thread 0 of the caller).
__device__ __forceinline__ void write_drift(const DriftAcc& t, int n, int64_t d, int have_master,
                                            DriftOut* out) {
    const double pairs = (double)n * (double)(n - 1) * 0.5;
    const double denom = (double)d * pairs;
    DriftOut r;
    r.max_abs = t.range;
    r.mean_sq = denom > 0.0 ? t.pair / denom : 0.0;
    r.rms = sqrt(r.mean_sq);
    r.mean_abs_to_master =
        have_master ? (d > 0 ? t.abs_sum / ((double)n * (double)d) : 0.0) : (double)NAN;
    r.stale_packets = t.stale;
    r.empty_packets = t.empty;
    *out = r;
}

// Device-coherent copies of a second-level partial (written by one
// workgroup, read by another that may sit on another XCD).
__device__ __forceinline__ void store_acc(DriftAcc* dst, const DriftAcc& a) {
    __hip_atomic_store(&dst->pair, a.pair, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&dst->abs_sum, a.abs_sum, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&dst->range, a.range, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&dst->stale, a.stale, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&dst->empty, a.empty, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ DriftAcc load_acc(const DriftAcc* src) {
    DriftAcc a;
    a.pair = __hip_atomic_load(&src->pair, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    a.abs_sum = __hip_atomic_load(&src->abs_sum, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    a.range = __hip_atomic_load(&src->range, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    a.stale = __hip_atomic_load(&src->stale, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    a.empty = __hip_atomic_load(&src->empty, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return a;
}

// Second level: kReduceGroups workgroups each fold a contiguous range of
// partials; the last workgroup to finish (by a counter that the kernel which
// wrote the partials zeroed) folds the kReduceGroups totals in a fixed order
// and writes the record.  Every sum has a fixed order, so the result does not
// depend on which workgroup finishes last.
__global__ __launch_bounds__(kThreads) void k_drift_reduce(const DriftPartial* parts, int64_t count,
                                                           DriftAcc* groups, int n, int64_t d,
                                                           int have_master, DriftOut* out) {
    __shared__ int s_last;
    unsigned* counter = reduce_counter(groups);
    const int64_t per = (count + kReduceGroups - 1) / kReduceGroups;
    const int64_t lo = (int64_t)blockIdx.x * per;
    const int64_t hi = lo + per < count ? lo + per : count;
    DriftAcc a;
    a.zero();
    int64_t j = lo + threadIdx.x;
    for (; j + 3 * kThreads < hi; j += 4 * kThreads) {
        DriftPartial q[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) q[u] = parts[j + u * kThreads];
#pragma unroll
        for (int u = 0; u < 4; ++u) a.add(q[u]);
    }
    for (; j < hi; j += kThreads) a.add(parts[j]);
    const DriftAcc t = block_fold<kThreads>(a);
    if (threadIdx.x == 0) {
        store_acc(groups + blockIdx.x, t);
        s_last = count_done(counter) == gridDim.x - 1;
    }
    __syncthreads();
    if (!s_last) return;
    DriftAcc b;
    b.zero();
    for (int g = threadIdx.x; g < kReduceGroups; g += kThreads) b.add(load_acc(groups + g));
    const DriftAcc tot = block_fold<kThreads>(b);
    if (threadIdx.x == 0) write_drift(tot, n, d, have_master, out);
}

// Up to kDirectFold partials: one workgroup of kFoldThreads folds them
// directly, in a fixed order, each thread with kFoldDepth loads in flight, so
// that up to kFoldThreads * kFoldDepth partials (the N = 8 step's 8192) take
// one memory round trip.
constexpr int kFoldThreads = 512;
constexpr int kFoldDepth = 16;
constexpr int64_t kDirectFold = 16384;

__global__ __launch_bounds__(kFoldThreads) void k_drift_direct(const DriftPartial* parts,
                                                               int64_t count, int n, int64_t d,
                                                               int have_master, DriftOut* out) {
    DriftAcc a;
    a.zero();
    // thread t folds partials j = t, t + kFoldThreads, ... in order; each
    // batch of kFoldDepth partials is requested (two 16-byte loads each; the
    // partials are 32 bytes, 32-byte aligned) before any is used
    static_assert(sizeof(DriftPartial) == 32, "two 16-byte loads per partial");
    union Raw {
        u32x4 v[2];
        DriftPartial q;
    };
    const u32x4* pv = reinterpret_cast<const u32x4*>(parts);
    int64_t j = threadIdx.x;
    for (; j + (kFoldDepth - 1) * kFoldThreads < count; j += kFoldDepth * kFoldThreads) {
        Raw q[kFoldDepth];
#pragma unroll
        for (int u = 0; u < kFoldDepth; ++u) {
            q[u].v[0] = pv[2 * (j + u * kFoldThreads)];
            q[u].v[1] = pv[2 * (j + u * kFoldThreads) + 1];
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < kFoldDepth; ++u) a.add(q[u].q);
    }
    for (; j < count; j += kFoldThreads) a.add(parts[j]);
    const DriftAcc t = block_fold<kFoldThreads>(a);
    if (threadIdx.x == 0) write_drift(t, n, d, have_master, out);
}

static hipError_t launch_drift_reduce(const DriftPartial* parts, int64_t count, DriftAcc* groups,
                                      int n, int64_t d, int have_master, DriftOut* out,
                                      hipStream_t s) {
    if (count <= kDirectFold) {
        hipLaunchKernelGGL(k_drift_direct, dim3(1), dim3(kFoldThreads), 0, s, parts, count, n, d,
                           have_master, out);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(k_drift_reduce, dim3(kReduceGroups), dim3(kThreads), 0, s, parts, count,
                       groups, n, d, have_master, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// The fused step: masks, aggregate, update, broadcast and drift partials in
// one pass.  HBM traffic per packet: the arrived gradient rows (read once),
// theta/m/v (read and written once), the arrived replica rows (written
// once) and, with drift, the stale replica rows (read once).
// ---------------------------------------------------------------------------
// The per-element part of one tile of the fused step (threads with nv > 0):
// aggregate, update, broadcast and, with DRIFT, the stale rows' drift sums.
template <class G, class R, bool DRIFT, bool W, class Pace>
__device__ __forceinline__ void step_chunk(const FusedParams& p, const Chunk& ch, const Pace& pace,
                                           const uint64_t (*s_words)[kMaxWords], int nw, int K,
                                           int RC, const Raw8<F32>& th_r, const Raw8<F32>& m_r,
                                           const Raw8<F32>& v_r, double& pair, double& range,
                                           double& abs_sum) {
    const bool relp = p.var.reliable != nullptr && p.var.reliable[ch.k] != 0;
    AggVariant var = p.var;
    if (var.parity_group > 0 && !relp) var.invq = parity_invq(var, ch.k, p.P);
    if (var.ge_derived && !relp) var.invq = ge_invq(var, p.step, ch.k, p.P);
    float th[8], mm[8], vv[8], g[8];
    unpack(th_r, th);
    aggregate8<G, W>(reinterpret_cast<const typename G::T*>(p.grads), p.ld_g, ch, s_words[0], p.n,
                     K, p.lam, th, var, relp, pace, g);
    if (p.opt.kind >= 1) unpack(m_r, mm);
    if (p.opt.kind == 2) unpack(v_r, vv);
    update8(p.opt, th, mm, vv, g);
    store_f32x8<W>(p.theta + ch.e0, ch.nv, th);
    if (p.opt.kind >= 1) store_f32x8<W>(p.m + ch.e0, ch.nv, mm);
    if (p.opt.kind == 2) store_f32x8<W>(p.v + ch.e0, ch.nv, vv);

    Packed8<R> r;
    r.pack(th);
    typename R::T* reps = reinterpret_cast<typename R::T*>(p.replicas);
    const int last_bits = p.n - (nw - 1) * 64;
    for (int w = 0; w < nw; ++w) {
        const uint64_t valid = (w == nw - 1 && last_bits < 64) ? ((1ull << last_bits) - 1) : ~0ull;
        uint64_t bits = uniform64(s_words[1][w]) & valid;
        while (bits) {
            const int i = w * 64 + __builtin_ctzll(bits);
            bits &= bits - 1;
            pace.rep(i);
            r.template store<W>(reps + (int64_t)i * p.ld_r + ch.e0, ch.nv);
        }
    }
    if (!DRIFT) return;
    // Stale rows (broadcast lost) in ascending order, after every store.
    Drift8<typename StepBounds8<R>::type> acc;
    float rv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) rv[j] = r.value(j);
    acc.init(RC > 0, rv);
    RowWalk stale(s_words[1], p.n, true, -1);
    stream_rows<RingDepth<Pace>::stale, R, W>(
        reps, p.ld_r, ch, stale, [&](int row) { pace.stale(row); },
        [&](const Raw8<R>& raw) {
            float x[8];
            unpack(raw, x);
            acc.add(x, rv, ch.nv);
        });
    acc.finish(p.n, ch.nv, pair, range);
    abs_sum = acc.abs_sum;
}

// One tile (a chunk of one packet) of the fused step in access form W.  The
// master and moments are requested before the masks are staged, so their
// latency overlaps the mask draws.
template <class G, class R, bool DRIFT, bool W, class Pace>
__device__ __forceinline__ void step_tile_w(const FusedParams& p, const Chunk& ch, int64_t tile,
                                            Pace pace, uint64_t (*s_words)[kMaxWords]) {
    constexpr int NT = R::kPacketThreads;
    Raw8<F32> th_r, m_r, v_r;
    if (ch.nv > 0) {
        load_raw<W>(p.theta + ch.e0, ch.nv, th_r);
        if (p.opt.kind >= 1) load_raw<W>(p.m + ch.e0, ch.nv, m_r);
        if (p.opt.kind == 2) load_raw<W>(p.v + ch.e0, ch.nv, v_r);
    }
    const int dirs[2] = {0, 1};
    stage_masks<NT, 2>(p.src, p.n, p.P, ch.k, p.step, dirs, s_words,
                       [&pace]() { pace.fetch(); });
    pace.begin();
    const int nw = (p.n + 63) >> 6;
    const int K = popcount_words(s_words[0], nw);
    const int RC = popcount_words(s_words[1], nw);

    if (ch.c == 0) {
        if (threadIdx.x == 0 && p.counts) p.counts[ch.k] = K;
        for (int i = threadIdx.x; i < p.n; i += NT) {
            const int64_t at = (int64_t)i * p.P + ch.k;
            const uint8_t rb = (s_words[1][i >> 6] >> (i & 63)) & 1;
            if (p.out_g) p.out_g[at] = (s_words[0][i >> 6] >> (i & 63)) & 1;
            if (p.out_b) p.out_b[at] = rb;
            if (p.ages) p.ages[at] = rb ? 0 : (p.ages[at] == 0xFFFF ? 0xFFFF : p.ages[at] + 1);
        }
    }

    double pair = 0.0, range = 0.0, abs_sum = 0.0;
    if (ch.nv > 0)
        step_chunk<G, R, DRIFT, W>(p, ch, pace, s_words, nw, K, RC, th_r, m_r, v_r, pair, range,
                                   abs_sum);
    if (DRIFT) {
        const uint32_t stale = ch.c == 0 ? (uint32_t)(p.n - RC) : 0u;
        const uint32_t empty = (ch.c == 0 && K == 0) ? 1u : 0u;
        block_reduce_partial<NT>(pair, abs_sum, range, stale, empty, p.partials + tile);
        if (tile == 0 && threadIdx.x == 0) *reduce_counter(p.groups) = 0u;
    }
}

// One tile (a chunk of one packet) of the fused step.  All NT threads of the
// workgroup call it; it stages the tile's masks in s_words (ending with a
// barrier).  `pace` delays row accesses (NoPace: none); it never changes
// what is computed.
template <class G, class R, bool DRIFT, class Pace>
__device__ __forceinline__ void step_tile(const FusedParams& p, int64_t tile, const Pace& pace,
                                          uint64_t (*s_words)[kMaxWords]) {
    constexpr int NT = R::kPacketThreads;
    const Chunk ch = chunk_at<NT>(tile, p.d, p.L, p.cpp);
    if (ch.whole) step_tile_w<G, R, DRIFT, true>(p, ch, tile, pace, s_words);
    else step_tile_w<G, R, DRIFT, false>(p, ch, tile, pace, s_words);
}

// One tile per workgroup.
template <class G, class R, bool DRIFT>
__global__ __launch_bounds__(R::kPacketThreads) void k_step_fused(FusedParams p) {
    __shared__ uint64_t s_words[2][kMaxWords];
    step_tile<G, R, DRIFT>(p, blockIdx.x, NoPace(), s_words);
}

// Anchor of the paced step's schedule: the clock time its first round
// starts, written by a one-lane kernel launched just before the step.  One
// anchor per device; overlapping paced steps on one device may read each
// other's anchor, which can cost speed but never changes a result.
__device__ uint64_t g_pace_anchor;

__global__ void k_pace_anchor(uint64_t margin_ticks) {
    if (threadIdx.x == 0)
        __hip_atomic_store(&g_pace_anchor, clock_ticks() + margin_ticks, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// Paced step: one tile per workgroup as in k_step_fused, tile b in round
// b / per_round, per_round no more than the workgroups the chip holds at
// once.  Round r's row accesses follow the slot schedule anchored at
// g_pace_anchor + r * round; the workgroups of round r + 1 take the places
// of round r's as those finish, around the time their own round starts.  A
// round covers adjacent tiles, so at any slot the chip streams a few long
// runs of one row instead of scattered pieces of every row.
template <class G, class R, bool DRIFT>
__global__ __launch_bounds__(R::kPacketThreads) void k_step_paced(FusedParams p, PaceParams q) {
    __shared__ uint64_t s_words[2][kMaxWords];
    __shared__ uint64_t s_anchor;  // read after the barrier that ends the mask staging
    ClockPace pace;
    pace.anchor_src = &g_pace_anchor;
    pace.anchor = &s_anchor;
    pace.round_start = (((uint64_t)blockIdx.x / (uint64_t)q.per_round) * q.round) >> 8;
    pace.off_g = q.off_g;
    pace.off_r = q.off_r;
    pace.off_s = q.off_s;
    pace.dg = q.dg;
    pace.dr = q.dr;
    pace.ds = q.ds;
    pace.guard = q.guard;
    step_tile<G, R, DRIFT>(p, blockIdx.x, pace, s_words);
}

// ---------------------------------------------------------------------------
// Persistent paced step for the plain configuration: arrived-mean estimator,
// no forced arrivals, ages or mask outputs, both directions' masks already in
// memory, whole tiles only (packet length and shard a multiple of 8).
// per_round workgroups loop over the rounds, workgroup b doing tile
// r * per_round + b in round r, so no workgroup starts or leaves between
// rounds.  The tile body is its own (no variant paths), so the loop carries
// nothing but the loop itself.
// ---------------------------------------------------------------------------
template <int NT>
__device__ __forceinline__ void stage_masks_mem2(const uint8_t* mem_g, const uint8_t* mem_b,
                                                 int n, int64_t P, int64_t k,
                                                 const ClockPace& pace,
                                                 uint64_t (*words)[kMaxWords]) {
    const int span = ((n + 63) >> 6) * 64;
    for (int base = 0; base < span; base += NT) {
        const int i = base + (int)threadIdx.x;
        const bool live = i < n;
        const int64_t at = (int64_t)(live ? i : n - 1) * P + k;
        const uint8_t bg = mem_g[at], bb = mem_b[at];
        if (base == 0) pace.fetch();
        if (i < span) {
            const uint64_t wg = __ballot(live && bg != 0);
            const uint64_t wb = __ballot(live && bb != 0);
            if ((threadIdx.x & 63) == 0) {
                words[0][i >> 6] = wg;
                words[1][i >> 6] = wb;
            }
        }
    }
    __syncthreads();
}

template <class G, class R, bool DRIFT>
__device__ __forceinline__ void lean_tile(const FusedParams& p, int64_t tile, ClockPace& pace,
                                          uint64_t (*s_words)[kMaxWords]) {
    constexpr int NT = R::kPacketThreads;
    const Chunk ch = chunk_at<NT>(tile, p.d, p.L, p.cpp);
    Raw8<F32> th_r, m_r, v_r;
    if (ch.nv > 0) {
        load_chunk<true>(p.theta, ch, th_r);
        if (p.opt.kind >= 1) load_chunk<true>(p.m, ch, m_r);
        if (p.opt.kind == 2) load_chunk<true>(p.v, ch, v_r);
    }
    stage_masks_mem2<NT>(p.src[0].mem, p.src[1].mem, p.n, p.P, ch.k, pace, s_words);
    pace.begin();
    const int nw = (p.n + 63) >> 6;
    const int K = popcount_words(s_words[0], nw);
    const int RC = popcount_words(s_words[1], nw);
    if (ch.c == 0 && threadIdx.x == 0 && p.counts) p.counts[ch.k] = K;
    double pair = 0.0, range = 0.0, abs_sum = 0.0;
    if (ch.nv > 0) {
        float th[8], mm[8], vv[8], g[8];
        unpack(th_r, th);
#pragma unroll
        for (int j = 0; j < 8; ++j) g[j] = 0.0f;
        RowWalk walk(s_words[0], p.n, false, -1);
        stream_rows<RingDepth<ClockPace>::grad, G, true>(
            reinterpret_cast<const typename G::T*>(p.grads), p.ld_g, ch, walk,
            [&](int row) { pace.grad(row); },
            [&](const Raw8<G>& raw) {
                float x[8];
                unpack(raw, x);
#pragma unroll
                for (int j = 0; j < 8; ++j) g[j] += x[j];
            });
        if (K > 0) {
            const float kf = (float)K;
#pragma unroll
            for (int j = 0; j < 8; ++j) g[j] = g[j] / kf;
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) g[j] = p.lam * th[j];
        }
        if (p.opt.kind >= 1) unpack(m_r, mm);
        if (p.opt.kind == 2) unpack(v_r, vv);
        update8(p.opt, th, mm, vv, g);
        store_chunk<true>(p.theta, ch, th);
        if (p.opt.kind >= 1) store_chunk<true>(p.m, ch, mm);
        if (p.opt.kind == 2) store_chunk<true>(p.v, ch, vv);
        Packed8<R> r;
        r.pack(th);
        typename R::T* reps = reinterpret_cast<typename R::T*>(p.replicas);
        RowWalk arrived(s_words[1], p.n, false, -1);
        for (int i = arrived.next(); i >= 0; i = arrived.next()) {
            pace.rep(i);
            store_chunk<true>(reps + (int64_t)i * p.ld_r, ch, r);
        }
        if (DRIFT) {
            Drift8<typename StepBounds8<R>::type> acc;
            float rv[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) rv[j] = r.value(j);
            acc.init(RC > 0, rv);
            RowWalk stale(s_words[1], p.n, true, -1);
            stream_rows<RingDepth<ClockPace>::stale, R, true>(
                reps, p.ld_r, ch, stale, [&](int row) { pace.stale(row); },
                [&](const Raw8<R>& raw) {
                    float x[8];
                    unpack(raw, x);
                    acc.add(x, rv, ch.nv);
                });
            acc.finish(p.n, ch.nv, pair, range);
            abs_sum = acc.abs_sum;
        }
    }
    if (DRIFT) {
        const uint32_t stale = ch.c == 0 ? (uint32_t)(p.n - RC) : 0u;
        const uint32_t empty = (ch.c == 0 && K == 0) ? 1u : 0u;
        block_reduce_partial<NT>(pair, abs_sum, range, stale, empty, p.partials + tile);
        if (tile == 0 && threadIdx.x == 0) *reduce_counter(p.groups) = 0u;
    }
}

template <class G, class R, bool DRIFT>
__global__ __launch_bounds__(R::kPacketThreads) void k_step_lean(FusedParams p, PaceParams q,
                                                                 int64_t tiles) {
    __shared__ uint64_t s_words[2][kMaxWords];
    __shared__ uint64_t s_anchor;
    for (int64_t r = 0;; ++r) {
        const int64_t tile = r * q.per_round + (int64_t)blockIdx.x;
        if (tile >= tiles) break;
        ClockPace pace;
        pace.anchor_src = &g_pace_anchor;
        pace.anchor = &s_anchor;
        pace.round_start = ((uint64_t)r * q.round) >> 8;
        pace.off_g = q.off_g;
        pace.off_r = q.off_r;
        pace.off_s = q.off_s;
        pace.dg = q.dg;
        pace.dr = q.dr;
        pace.ds = q.ds;
        pace.guard = q.guard;
        lean_tile<G, R, DRIFT>(p, tile, pace, s_words);
        // the next tile rewrites the masks and the anchor in LDS
        __syncthreads();
    }
}

__global__ void k_drift_zero(DriftOut* out) {
    if (threadIdx.x == 0) {
        DriftOut r;
        r.max_abs = 0.0;
        r.mean_sq = 0.0;
        r.rms = 0.0;
        r.mean_abs_to_master = 0.0;
        r.stale_packets = 0;
        r.empty_packets = 0;
        *out = r;
    }
}

// ---------------------------------------------------------------------------
// Launchers (host)
// ---------------------------------------------------------------------------
static int64_t grid_cap(int64_t blocks) { return blocks < (1ll << 20) ? blocks : (1ll << 20); }

hipError_t launch_masks_bernoulli(int n, int64_t num_packets, uint64_t step, int dir,
                                  uint64_t seed, uint64_t thr, int owner,
                                  const uint8_t* reliable, uint8_t* arrived, hipStream_t s) {
    const int64_t total = (int64_t)n * num_packets;
    const int64_t blocks = grid_cap((total + kThreads - 1) / kThreads);
    hipLaunchKernelGGL(k_masks_bernoulli, dim3((unsigned)blocks), dim3(kThreads), 0, s, n,
                       num_packets, step, (uint64_t)dir, seed, thr, owner, reliable, arrived);
    return hipGetLastError();
}

hipError_t launch_masks_bernoulli_jobs(int n, int64_t num_packets, uint64_t step,
                                       const MaskJob* jobs, int njobs, hipStream_t s) {
    MaskJobs J;
    for (int j = 0; j < njobs; ++j) J.job[j] = jobs[j];
    const int64_t total = (int64_t)n * num_packets * njobs;
    const int64_t blocks = grid_cap((total + kThreads - 1) / kThreads);
    hipLaunchKernelGGL(k_masks_bernoulli_jobs, dim3((unsigned)blocks), dim3(kThreads), 0, s, n,
                       num_packets, step, njobs, J);
    return hipGetLastError();
}

hipError_t launch_masks_parity(const ParityLaunch& L, hipStream_t s) {
    const int64_t blocks = (int64_t)L.ndir * L.n * L.spans;
    hipLaunchKernelGGL(k_masks_parity, dim3((unsigned)blocks), dim3(kThreads), 0, s, L);
    return hipGetLastError();
}

__global__ __launch_bounds__(kThreads) void k_ages_update(int64_t total, const uint8_t* arrived,
                                                          uint16_t* ages) {
    for (int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * kThreads) {
        const uint16_t a = ages[idx];
        ages[idx] = arrived[idx] ? 0 : (a == 0xFFFF ? 0xFFFF : a + 1);
    }
}

hipError_t launch_ages_update(int64_t total, const uint8_t* arrived, uint16_t* ages,
                              hipStream_t s) {
    const int64_t blocks = grid_cap((total + kThreads - 1) / kThreads);
    hipLaunchKernelGGL(k_ages_update, dim3((unsigned)blocks), dim3(kThreads), 0, s, total, arrived,
                       ages);
    return hipGetLastError();
}

hipError_t launch_masks_ge(const GeLaunch& L, int ndir, hipStream_t s) {
    const int64_t blocks = (int64_t)ndir * L.n * L.S;
    hipLaunchKernelGGL(k_ge_compose, dim3((unsigned)blocks), dim3(kThreads), 0, s, L);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_ge_apply, dim3((unsigned)blocks), dim3(kThreads), 0, s, L);
    return hipGetLastError();
}

// Chunks per packet and workgroups for a per-packet kernel of NT threads.
template <int NT>
static int64_t packet_grid(int64_t P, int64_t L, int* cpp) {
    *cpp = (int)((L + NT * kElems - 1) / (NT * kElems));
    return P * *cpp;
}

template <class G>
static void launch_aggregate_t(AggParams p, hipStream_t s) {
    constexpr int NT = G::kPacketThreads;
    const int64_t blocks = packet_grid<NT>(p.P, p.L, &p.cpp);
    hipLaunchKernelGGL(k_aggregate<G>, dim3((unsigned)blocks), dim3(NT), 0, s, p);
}

hipError_t launch_aggregate(int gdtype, const AggParams& p, hipStream_t s) {
    if (gdtype == 1) launch_aggregate_t<BF16>(p, s);
    else launch_aggregate_t<F32>(p, s);
    return hipGetLastError();
}

hipError_t launch_shard_step(int64_t d, const OptParams& o, float* theta, float* m, float* v,
                             const float* g_hat, hipStream_t s) {
    const int64_t blocks = (d + kThreads * kElems - 1) / (kThreads * kElems);
    hipLaunchKernelGGL(k_shard_step, dim3((unsigned)blocks), dim3(kThreads), 0, s, d, o, theta,
                       m, v, g_hat);
    return hipGetLastError();
}

template <class R>
static void launch_broadcast_t(BcastParams p, hipStream_t s) {
    constexpr int NT = R::kPacketThreads;
    const int64_t blocks = packet_grid<NT>(p.P, p.L, &p.cpp);
    hipLaunchKernelGGL(k_broadcast<R>, dim3((unsigned)blocks), dim3(NT), 0, s, p);
}

hipError_t launch_broadcast(int rdtype, const BcastParams& p, hipStream_t s) {
    if (rdtype == 1) launch_broadcast_t<BF16>(p, s);
    else launch_broadcast_t<F32>(p, s);
    return hipGetLastError();
}

template <class R>
static int64_t launch_drift_t(DriftParams p, hipStream_t s) {
    constexpr int NT = R::kPacketThreads;
    const int64_t blocks = packet_grid<NT>(p.P, p.L, &p.cpp);
    hipLaunchKernelGGL(k_drift<R>, dim3((unsigned)blocks), dim3(NT), 0, s, p);
    return blocks;
}

hipError_t launch_drift(int rdtype, const DriftParams& p, int n, int64_t d, int have_master,
                        DriftOut* out, hipStream_t s) {
    const int64_t blocks = rdtype == 1 ? launch_drift_t<BF16>(p, s) : launch_drift_t<F32>(p, s);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_drift_reduce(p.partials, blocks, p.groups, n, d, have_master, out, s);
}

// ---------------------------------------------------------------------------
// Pacing of the fused step
// ---------------------------------------------------------------------------
namespace {
std::atomic<int> g_pace_mode{0};
std::atomic<double> g_pace_rate{kDefaultPaceRate};
std::atomic<double> g_pace_gap_us{kDefaultPaceGapUs};
std::atomic<double> g_pace_lead_us{kDefaultPaceLeadUs};
std::atomic<int> g_pace_overlap{kDefaultPaceOverlap};
std::atomic<int> g_pace_resident{kDefaultPaceResident};
std::atomic<double> g_pace_headroom{kDefaultPaceHeadroom};
std::atomic<double> g_pace_tail_us{kDefaultPaceTailUs};
std::atomic<int> g_pace_persistent{kDefaultPacePersistent};
std::atomic<double> g_pace_rate_f32{kDefaultPaceRateF32};

// Compute units and clock rate of a device, and resident workgroups per
// compute unit of a kernel, looked up once per device into fixed tables (no
// host allocation on the call path).
std::mutex g_cache_mu;
struct DevInfo {
    bool known;
    int cus;
    double tick_hz;
};
DevInfo g_dev_info[kMaxDevices];

bool device_info(int dev, int* cus, double* tick_hz) {
    if (dev < 0 || dev >= kMaxDevices) return false;
    std::lock_guard<std::mutex> lk(g_cache_mu);
    DevInfo& di = g_dev_info[dev];
    if (!di.known) {
        int c = 0, khz = 0;
        if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess)
            return false;
        di = DevInfo{true, c, 1e3 * (double)khz};
    }
    *cus = di.cus;
    *tick_hz = di.tick_hz;
    return *cus > 0 && *tick_hz > 0.0;
}

// Resident workgroups per compute unit of one kernel (one table per kernel:
// the caller passes a table of its own).
template <class K>
int resident_per_cu(int dev, K kernel, int threads, int (&table)[kMaxDevices]) {
    if (dev < 0 || dev >= kMaxDevices) return 0;
    std::lock_guard<std::mutex> lk(g_cache_mu);
    if (table[dev] == 0) {
        int nb = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kernel, threads, 0) != hipSuccess)
            nb = 0;
        table[dev] = nb > 0 ? nb : -1;
    }
    return table[dev] > 0 ? table[dev] : 0;
}
}  // namespace

PaceSetting get_pace_setting() {
    return PaceSetting{g_pace_mode.load(), g_pace_rate.load(), g_pace_gap_us.load(),
                       g_pace_lead_us.load(), g_pace_overlap.load(), g_pace_resident.load(),
                       g_pace_headroom.load(), g_pace_tail_us.load(), g_pace_persistent.load(),
                       g_pace_rate_f32.load()};
}

void set_pace_setting(const PaceSetting& st) {
    g_pace_mode.store(st.mode);
    g_pace_rate.store(st.bytes_per_s);
    g_pace_gap_us.store(st.gap_us);
    g_pace_lead_us.store(st.lead_us);
    g_pace_overlap.store(st.overlap);
    g_pace_resident.store(st.resident);
    g_pace_headroom.store(st.headroom);
    g_pace_tail_us.store(st.tail_us);
    g_pace_persistent.store(st.persistent);
    g_pace_rate_f32.store(st.bytes_per_s_f32);
}

// Lay out the schedule of a paced step with `tiles` tiles, or return false
// to run it unpaced.  `overlap` rounds stream at once, each covering *grid
// adjacent tiles (`resident` rounds fill at most kPaceHeadroom of the
// resident workgroup places; rounds are balanced) and laid out for its
// share, rate / overlap, of the bandwidth.  A round is: a
// lead for the workgroups to start, draw masks and read their master and
// moments; the gradient sweep; the gap for the update and the master and
// moment writes; the replica sweep; the stale-read sweep.  Each sweep's slot
// lasts as long as the rows that slot is expected to move take at the
// round's share.  Rounds start round / overlap apart, so with two in flight
// one round's gradient sweep runs beside the previous round's replica sweep
// and each round's lead, gap and tail are covered by the other's streams.
template <class G, class R, bool DRIFT>
static bool pace_plan(const PaceSetting& st, bool lean, const FusedParams& p, const PaceHint& h,
                      int64_t tiles, PaceParams* q, int64_t* grid, uint64_t* margin) {
    constexpr int NT = R::kPacketThreads;
    // Steps with fp32 replica rows (128-thread workgroups, two loads per row
    // and thread) keep their schedule at a lower rate than bf16 rows.
    const double rate = sizeof(typename R::T) == 4 ? st.bytes_per_s_f32 : st.bytes_per_s;
    if (st.mode == kPaceNever || !(rate > 0.0) || tiles <= 0) return false;
    int dev = 0, cus = 0;
    double tick_hz = 0.0;
    if (hipGetDevice(&dev) != hipSuccess || !device_info(dev, &cus, &tick_hz)) return false;
    static int occupancy[kMaxDevices], occupancy_lean[kMaxDevices];
    const int per_cu = lean ? resident_per_cu(dev, k_step_lean<G, R, DRIFT>, NT, occupancy_lean)
                            : resident_per_cu(dev, k_step_paced<G, R, DRIFT>, NT, occupancy);
    const int k = st.overlap < 1 ? 1 : (st.overlap > 2 ? 2 : st.overlap);
    const int res = st.resident < k ? k : st.resident;
    // A round of an fp32-row kernel is at most kPaceMaxRoundTiles tiles (a
    // row slot streams 4 MiB): rounds of every resident place of those
    // kernels (2048 tiles) were measured slower than rounds of half of them.
    // Rounds of the bf16-row kernels take every place (1280 with drift,
    // 1536 without): capped at 1024, the next round's workgroups start early
    // in the spare places and the schedule is not kept.
    int64_t gmax = (int64_t)(st.headroom * per_cu * cus / res);
    if (sizeof(typename R::T) == 4 && gmax > kPaceMaxRoundTiles) gmax = kPaceMaxRoundTiles;
    if (gmax < 1) return false;
    const int64_t rounds = (tiles + gmax - 1) / gmax;
    // Auto: only where pacing was measured to pay, many rows (the N = 64
    // steps gain 5-10%); a few rows break even or lose.
    if (st.mode == kPaceAuto && (rounds < kPaceMinRounds || p.n < kPaceMinRows)) return false;
    const int64_t g = (tiles + rounds - 1) / rounds;
    const double row_g = (double)NT * kElems * sizeof(typename G::T);
    const double row_r = (double)NT * kElems * sizeof(typename R::T);
    const double state = (double)NT * kElems * 4.0 * (p.opt.kind + 1);
    const double fp = 256.0 * tick_hz * k / rate;  // 1/256 ticks per byte of a round
    const double us = 1e-6 * tick_hz * 256.0;                 // 1/256 ticks per microsecond
    const double qg = h.q_g < 0.0 ? 0.0 : (h.q_g > 1.0 ? 1.0 : h.q_g);
    const double qb = h.q_b < 0.0 ? 0.0 : (h.q_b > 1.0 ? 1.0 : h.q_b);
    const double n = (double)p.n;
    const double dg = g * row_g * qg * fp;
    const double dr = g * row_r * qb * fp;
    const double ds = DRIFT ? g * row_r * (1.0 - qb) * fp : 0.0;
    const double off_g = st.lead_us * us + g * state * fp;
    const double off_r = off_g + n * dg + g * state * fp + st.gap_us * us;
    const double off_s = off_r + n * dr;
    // A round's workgroups leave a little after its last slot: the last rows
    // they read must arrive and the drift partial be folded.
    const double length = off_s + n * ds + st.tail_us * us;
    // Rounds start `spacing` apart: no closer than the round's bytes at its
    // share allow with k rounds streaming (stream / k), and far enough apart
    // that a round's workgroups find places when it starts, res rounds
    // sharing the resident places (length / res).  With k = 2 and res = 3
    // the lead, gap and tail of each round are covered by the other rounds'
    // streams.
    const double stream = n * (dg + dr + ds) + 2.0 * g * state * fp;
    const double spacing = stream / k > length / res ? stream / k : length / res;
    if (!(length < 1e15)) return false;
    q->per_round = g;
    q->dg = (uint64_t)dg;
    q->dr = (uint64_t)dr;
    q->ds = (uint64_t)ds;
    q->off_g = (uint64_t)off_g;
    q->off_r = (uint64_t)off_r;
    q->off_s = (uint64_t)off_s;
    q->round = (uint64_t)spacing;
    *margin = (uint64_t)(kPaceMarginUs * 1e-6 * tick_hz) + 1;
    q->guard = 2 * ((uint64_t)length >> 8) + 2 * *margin + 1;
    *grid = g;
    return true;
}

// The fused step's geometry follows the replica type, like the standalone
// drift kernel, so both fold drift partials over the same partition.
template <class G, class R, bool DRIFT>
static int64_t launch_fused_grd(const FusedParams& p, const PaceHint& h, hipStream_t s) {
    constexpr int NT = R::kPacketThreads;
    FusedParams pp = p;
    const int64_t tiles = packet_grid<NT>(pp.P, pp.L, &pp.cpp);
    PaceParams q;
    int64_t grid = 0;
    uint64_t margin = 0;
    const PaceSetting st = get_pace_setting();
    // Bernoulli masks drawn in the step would put every workgroup's draws at
    // the start of its round, all at once; a paced step has them drawn
    // beforehand by the mask kernel, where memory for them is at hand, and
    // reads them.
    FusedParams pm = pp;
    MaskJob jobs[2];
    int njobs = 0;
    for (int dir = 0; dir < 2; ++dir) {
        if (!pm.src[dir].draw || !pm.pre[dir]) continue;
        const MaskSource& m = pm.src[dir];
        jobs[njobs++] = MaskJob{(uint64_t)dir, m.seed, m.thr, m.owner, m.reliable, pm.pre[dir]};
        pm.src[dir] = MaskSource{false, 0, 0, pm.pre[dir], -1, nullptr};
        if (dir == 0 && pm.out_g == pm.pre[0]) pm.out_g = nullptr;
        if (dir == 1 && pm.out_b == pm.pre[1]) pm.out_b = nullptr;
    }
    // The persistent form takes the plain configuration only (see k_step_lean).
    bool lean = st.persistent && pm.var.kind == kEstArrivedMean && !pm.ages && !pm.out_g &&
                !pm.out_b && pm.L % 8 == 0 && pm.d % 8 == 0;
    for (int dir = 0; dir < 2; ++dir)
        lean = lean && !pm.src[dir].draw && pm.src[dir].owner < 0 && !pm.src[dir].reliable;
    if (pace_plan<G, R, DRIFT>(st, lean, pm, h, tiles, &q, &grid, &margin)) {
        if (njobs && launch_masks_bernoulli_jobs(pm.n, pm.P, pm.step, jobs, njobs, s) != hipSuccess)
            return -1;
        hipLaunchKernelGGL(k_pace_anchor, dim3(1), dim3(64), 0, s, margin);
        if (lean)
            hipLaunchKernelGGL((k_step_lean<G, R, DRIFT>), dim3((unsigned)grid), dim3(NT), 0, s,
                               pm, q, tiles);
        else
            hipLaunchKernelGGL((k_step_paced<G, R, DRIFT>), dim3((unsigned)tiles), dim3(NT), 0, s,
                               pm, q);
    } else {
        hipLaunchKernelGGL((k_step_fused<G, R, DRIFT>), dim3((unsigned)tiles), dim3(NT), 0, s, pp);
    }
    return tiles;
}

template <class G, class R>
static int64_t launch_fused_gr(bool drift, const FusedParams& p, const PaceHint& h,
                               hipStream_t s) {
    return drift ? launch_fused_grd<G, R, true>(p, h, s) : launch_fused_grd<G, R, false>(p, h, s);
}

hipError_t launch_fused(int gdtype, int rdtype, const FusedParams& p, DriftOut* drift,
                        const PaceHint& h, hipStream_t s) {
    const bool dr = drift != nullptr;
    int64_t blocks;
    if (gdtype == 1 && rdtype == 1) blocks = launch_fused_gr<BF16, BF16>(dr, p, h, s);
    else if (gdtype == 1) blocks = launch_fused_gr<BF16, F32>(dr, p, h, s);
    else if (rdtype == 1) blocks = launch_fused_gr<F32, BF16>(dr, p, h, s);
    else blocks = launch_fused_gr<F32, F32>(dr, p, h, s);
    if (blocks < 0) return hipErrorLaunchFailure;
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !dr) return e;
    return launch_drift_reduce(p.partials, blocks, p.groups, p.n, p.d, 1, drift, s);
}

hipError_t launch_drift_zero(DriftOut* out, hipStream_t s) {
    hipLaunchKernelGGL(k_drift_zero, dim3(1), dim3(64), 0, s, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Static scratch of the entry point that allocates nothing.  Each device that
// loads the library holds its own copy until the process ends; host code
// reaches it only through the device address that hipGetSymbolAddress gives
// on that device (the array's own name is not a device address on the host).
// ---------------------------------------------------------------------------
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];
}  // namespace

hipError_t noalloc_scratch(void** ptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace lossy
