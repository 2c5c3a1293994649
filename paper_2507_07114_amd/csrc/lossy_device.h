// Device-side building blocks of the lossy step for gfx950 (CDNA4, wave64).
//
// Every kernel of the library is assembled from the pieces in this header,
// so the fused step and the one-stage-at-a-time entry points run the same
// arithmetic in the same order and produce bit-identical results.  The
// library is compiled with -ffp-contract=off: every fused multiply-add below
// is written out explicitly.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lossy {

constexpr int kThreads = 256;  // threads per workgroup of the flat kernels (4 waves)
constexpr int kElems = 8;      // consecutive elements per thread
// Per-packet kernels size their workgroups by the element type of the rows
// they stream (F32::kPacketThreads, BF16::kPacketThreads): a workgroup then
// covers 4 KiB of each row, which measured fastest for both types.
constexpr int kMinPacketThreads = 128;
constexpr int kMaxWorkers = 1024;
constexpr int kMaxWords = kMaxWorkers / 64;
// Row loads in flight per thread while streaming the arrived gradient rows
// and the stale replica rows (a ring: the load of row j + depth is issued as
// soon as row j has been used) in an unpaced step, where a workgroup's own
// loads are all that keeps the memory busy.  The paced step's depth is
// RingDepth<ClockPace> below.
constexpr int kDepthGrad = 4;
constexpr int kDepthStale = 4;
// Gradient rows per batch of the stale-fill estimator, which reads every row.
constexpr int kBatchGrad = 4;
// Replica rows in flight per thread in the standalone drift pass, which reads
// every row: deeper batches cost occupancy (2.85 ms at 2 against 3.18 at 4 and
// 3.82 at 8 for the 64 x 105M bf16 replicas).
constexpr int kBatchDrift = 2;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds, each
// multiplying words 0 and 2 by fixed odd constants, exchanging the halves of
// the products with words 1 and 3 and the round key; the key is bumped by two
// Weyl constants between rounds.  Only output words 0 and 1 are needed.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2,
                                              uint64_t c3, uint64_t k0, uint64_t k1,
                                              uint64_t& w0, uint64_t& w1) {
    const uint64_t kM0 = 0xD2E7470EE14C6C93ull, kM1 = 0xCA5A826395121157ull;
    const uint64_t kW0 = 0x9E3779B97F4A7C15ull, kW1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += kW0;
            k1 += kW1;
        }
        const uint64_t hi0 = __umul64hi(kM0, c0), lo0 = kM0 * c0;
        const uint64_t hi1 = __umul64hi(kM1, c2), lo1 = kM1 * c2;
        const uint64_t n0 = hi1 ^ c1 ^ k0;
        const uint64_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
    }
    w0 = c0;
    w1 = c1;
}

// Arrival of (packet k, worker i, step t, direction dir) under i.i.d. loss:
// lost iff hi32(w0) < thr, thr = ceil(p * 2^32) (host-computed).
__device__ __forceinline__ bool bernoulli_arrived(uint64_t k, uint64_t i, uint64_t t,
                                                  uint64_t dir, uint64_t seed,
                                                  uint64_t thr) {
    uint64_t w0, w1;
    philox4x64_10(k, i, t, dir, seed, 0, w0, w1);
    return (w0 >> 32) >= thr;
}

// ---------------------------------------------------------------------------
// Element types.  bf16 is carried as its 16-bit pattern (the upper half of a
// binary32); narrowing rounds to nearest even, NaN stays quiet NaN.
// ---------------------------------------------------------------------------
struct F32 {
    typedef float T;
    static constexpr int kPacketThreads = 128;
};
struct BF16 {
    typedef uint16_t T;
    static constexpr int kPacketThreads = 256;
};

__device__ __forceinline__ float bf16_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Memory access of a thread's 8 consecutive elements.  Kernels decide per
// tile (wave-uniformly) which of two forms every access of the tile takes:
//   W = true   every thread of the tile owns 0 or 8 elements and the tile
//              starts on a 16-byte boundary: one 16-byte access per 8 bf16
//              (two per 8 fp32), predicated on nv == 8.  Loads land in raw
//              registers and are unpacked only when used, so a batch of row
//              loads is in flight together.
//   W = false  element by element (a shard end that is not a multiple of 8,
//              or packets whose length is not a multiple of 8 elements).
// Raw storage of 8 consecutive elements.
template <class E>
struct Raw8;
template <>
struct Raw8<F32> {
    u32x4 a, b;
};
template <>
struct Raw8<BF16> {
    u32x4 a;
};

template <bool W>
__device__ __forceinline__ void load_raw(const float* p, int nv, Raw8<F32>& r) {
    r.a = u32x4{0, 0, 0, 0};
    r.b = u32x4{0, 0, 0, 0};
    if (W) {
        if (nv == 8) {
            r.a = *reinterpret_cast<const u32x4*>(p);
            r.b = *reinterpret_cast<const u32x4*>(p + 4);
        }
    } else {
        uint32_t w[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) w[j] = j < nv ? __float_as_uint(p[j]) : 0u;
        r.a = u32x4{w[0], w[1], w[2], w[3]};
        r.b = u32x4{w[4], w[5], w[6], w[7]};
    }
}

template <bool W>
__device__ __forceinline__ void load_raw(const uint16_t* p, int nv, Raw8<BF16>& r) {
    r.a = u32x4{0, 0, 0, 0};
    if (W) {
        if (nv == 8) r.a = *reinterpret_cast<const u32x4*>(p);
    } else {
        uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
        for (int j = 0; j < 8; ++j)
            if (j < nv) w[j >> 1] |= (uint32_t)p[j] << (16 * (j & 1));
        r.a = u32x4{w[0], w[1], w[2], w[3]};
    }
}

__device__ __forceinline__ void unpack(const Raw8<F32>& r, float (&x)[8]) {
    x[0] = __uint_as_float(r.a.x); x[1] = __uint_as_float(r.a.y);
    x[2] = __uint_as_float(r.a.z); x[3] = __uint_as_float(r.a.w);
    x[4] = __uint_as_float(r.b.x); x[5] = __uint_as_float(r.b.y);
    x[6] = __uint_as_float(r.b.z); x[7] = __uint_as_float(r.b.w);
}

__device__ __forceinline__ void unpack(const Raw8<BF16>& r, float (&x)[8]) {
    x[0] = bf16_to_f32(r.a.x & 0xFFFFu); x[1] = bf16_to_f32(r.a.x >> 16);
    x[2] = bf16_to_f32(r.a.y & 0xFFFFu); x[3] = bf16_to_f32(r.a.y >> 16);
    x[4] = bf16_to_f32(r.a.z & 0xFFFFu); x[5] = bf16_to_f32(r.a.z >> 16);
    x[6] = bf16_to_f32(r.a.w & 0xFFFFu); x[7] = bf16_to_f32(r.a.w >> 16);
}

// 8 consecutive elements as floats (0 past nv).
template <class E, bool W>
__device__ __forceinline__ void load8(const typename E::T* p, int nv, float (&x)[8]) {
    Raw8<E> r;
    load_raw<W>(p, nv, r);
    unpack(r, x);
}

// Rounded storage form of 8 values (what a replica row holds).
template <class E>
struct Packed8;

template <>
struct Packed8<F32> {
    Raw8<F32> r;
    __device__ __forceinline__ void pack(const float (&x)[8]) {
        r.a = u32x4{__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]),
                    __float_as_uint(x[3])};
        r.b = u32x4{__float_as_uint(x[4]), __float_as_uint(x[5]), __float_as_uint(x[6]),
                    __float_as_uint(x[7])};
    }
    __device__ __forceinline__ float value(int j) const {
        const u32x4& h = j < 4 ? r.a : r.b;
        const int q = j & 3;
        return __uint_as_float(q == 0 ? h.x : q == 1 ? h.y : q == 2 ? h.z : h.w);
    }
    template <bool W>
    __device__ __forceinline__ void store(float* p, int nv) const {
        if (W) {
            if (nv == 8) {
                __builtin_nontemporal_store(r.a, reinterpret_cast<u32x4*>(p));
                __builtin_nontemporal_store(r.b, reinterpret_cast<u32x4*>(p + 4));
            }
        } else {
            for (int j = 0; j < nv; ++j) p[j] = value(j);
        }
    }
};

template <>
struct Packed8<BF16> {
    Raw8<BF16> r;
    __device__ __forceinline__ void pack(const float (&x)[8]) {
        r.a = u32x4{f32_to_bf16(x[0]) | (f32_to_bf16(x[1]) << 16),
                    f32_to_bf16(x[2]) | (f32_to_bf16(x[3]) << 16),
                    f32_to_bf16(x[4]) | (f32_to_bf16(x[5]) << 16),
                    f32_to_bf16(x[6]) | (f32_to_bf16(x[7]) << 16)};
    }
    __device__ __forceinline__ float value(int j) const {
        const int q = j >> 1;
        const uint32_t w = q == 0 ? r.a.x : q == 1 ? r.a.y : q == 2 ? r.a.z : r.a.w;
        return bf16_to_f32((j & 1) ? (w >> 16) : (w & 0xFFFFu));
    }
    template <bool W>
    __device__ __forceinline__ void store(uint16_t* p, int nv) const {
        if (W) {
            if (nv == 8) __builtin_nontemporal_store(r.a, reinterpret_cast<u32x4*>(p));
        } else {
            for (int j = 0; j < nv; ++j) p[j] = (uint16_t)f32_to_bf16(value(j));
        }
    }
};

template <bool W>
__device__ __forceinline__ void store_f32x8(float* p, int nv, const float (&x)[8]) {
    if (W) {
        if (nv == 8) {
            *reinterpret_cast<u32x4*>(p) = u32x4{__float_as_uint(x[0]), __float_as_uint(x[1]),
                                                 __float_as_uint(x[2]), __float_as_uint(x[3])};
            *reinterpret_cast<u32x4*>(p + 4) = u32x4{__float_as_uint(x[4]), __float_as_uint(x[5]),
                                                     __float_as_uint(x[6]), __float_as_uint(x[7])};
        }
    } else {
        for (int j = 0; j < nv; ++j) p[j] = x[j];
    }
}

// Store raw storage back bit for bit (16-byte non-temporal stores when W).
template <bool W>
__device__ __forceinline__ void store_raw(float* p, int nv, const Raw8<F32>& r) {
    if (W) {
        if (nv == 8) {
            __builtin_nontemporal_store(r.a, reinterpret_cast<u32x4*>(p));
            __builtin_nontemporal_store(r.b, reinterpret_cast<u32x4*>(p + 4));
        }
    } else {
        const uint32_t w[8] = {r.a.x, r.a.y, r.a.z, r.a.w, r.b.x, r.b.y, r.b.z, r.b.w};
        for (int j = 0; j < nv; ++j) p[j] = __uint_as_float(w[j]);
    }
}

template <bool W>
__device__ __forceinline__ void store_raw(uint16_t* p, int nv, const Raw8<BF16>& r) {
    if (W) {
        if (nv == 8) __builtin_nontemporal_store(r.a, reinterpret_cast<u32x4*>(p));
    } else {
        const uint32_t w[4] = {r.a.x, r.a.y, r.a.z, r.a.w};
        for (int j = 0; j < nv; ++j) p[j] = (uint16_t)(w[j >> 1] >> (16 * (j & 1)));
    }
}

// ---------------------------------------------------------------------------
// Row loads through a buffer resource (CDNA buffer instructions).  The
// resource of a row's chunk has the chunk's valid bytes as its size, so a
// lane past the data reads zeros without touching memory, and a resource of
// size 0 gives a load that moves nothing.  Streaming loops issue such a load
// unconditionally on every lane, so each iteration has the same number of
// loads in flight and the compiler waits for one row at a time instead of
// draining every load.
// ---------------------------------------------------------------------------
constexpr int kBufferWord3 = 0x00020000;  // gfx9-family word 3: 32-bit data format

__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void* base, int bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes,
                                             kBufferWord3);
}

__device__ __forceinline__ void load_buf(__amdgpu_buffer_rsrc_t r, int lane_bytes, Raw8<BF16>& x) {
    x.a = __builtin_amdgcn_raw_buffer_load_b128(r, lane_bytes, 0, 0);
}

__device__ __forceinline__ void load_buf(__amdgpu_buffer_rsrc_t r, int lane_bytes, Raw8<F32>& x) {
    x.a = __builtin_amdgcn_raw_buffer_load_b128(r, lane_bytes, 0, 0);
    x.b = __builtin_amdgcn_raw_buffer_load_b128(r, lane_bytes + 16, 0, 0);
}

// Wave-uniform copy of a 64-bit value held identically by all active lanes.
__device__ __forceinline__ uint64_t uniform64(uint64_t x) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// ---------------------------------------------------------------------------
// Per-packet masks in LDS: word w bit b = arrival of worker 64 w + b.
// ---------------------------------------------------------------------------
struct MaskSource {
    // draw == true: Bernoulli draw in the kernel with (seed, thr);
    // otherwise read bytes from mem[i * num_packets + k].
    bool draw;
    uint64_t seed, thr;
    const uint8_t* mem;
    // Transfers that cannot be lost: row `owner` (-1 none) and packets with
    // reliable[k] = 1 (reliable may be null) always arrive.
    int owner;
    const uint8_t* reliable;
};

__device__ __forceinline__ bool forced_arrival(int i, int64_t k, int owner,
                                               const uint8_t* reliable) {
    return i == owner || (reliable != nullptr && reliable[k] != 0);
}

// Stage the masks of packet k for NDIR directions into words[s][w]
// (direction dirs[s] drawn from src[s]).  All NT threads of the workgroup must
// call it (it ends with a barrier).  The source of each direction is indexed
// by a compile-time constant, so its fields are read once per workgroup, and
// the mask bytes of every direction are requested before any is used;
// `fetch()` is called once by every thread right after the first requests,
// so a load of its own overlaps them.
struct NoFetch {
    __device__ __forceinline__ void operator()() const {}
};

template <int NT, int NDIR, class Fetch = NoFetch>
__device__ __forceinline__ void stage_masks(const MaskSource* src, int n, int64_t num_packets,
                                            int64_t k, uint64_t step, const int* dirs,
                                            uint64_t (*words)[kMaxWords],
                                            const Fetch& fetch = Fetch()) {
    const int nw = (n + 63) >> 6;
    const int span = nw * 64;
    bool rel[NDIR];
#pragma unroll
    for (int s = 0; s < NDIR; ++s) rel[s] = src[s].reliable != nullptr && src[s].reliable[k] != 0;
    bool all_mem = true;
#pragma unroll
    for (int s = 0; s < NDIR; ++s) all_mem = all_mem && !src[s].draw;
    auto part = [&](int base) {
        const int i = base + (int)threadIdx.x;
        const bool live = i < n;
        // lanes past the last worker read worker n - 1's byte and ignore it,
        // so that every lane issues the same loads
        const int64_t at = (int64_t)(live ? i : n - 1) * num_packets + k;
        uint8_t byte[NDIR];
        if (all_mem) {
#pragma unroll
            for (int s = 0; s < NDIR; ++s) byte[s] = src[s].mem[at];
        } else {
#pragma unroll
            for (int s = 0; s < NDIR; ++s) byte[s] = src[s].draw ? 0 : src[s].mem[at];
        }
        if (base == 0) fetch();
        bool arrived[NDIR];
#pragma unroll
        for (int s = 0; s < NDIR; ++s) {
            bool a = false;
            if (live) {
                a = src[s].draw ? bernoulli_arrived((uint64_t)k, (uint64_t)i, step,
                                                    (uint64_t)dirs[s], src[s].seed, src[s].thr)
                                : byte[s] != 0;
                a = a || i == src[s].owner || rel[s];
            }
            arrived[s] = a;
        }
        // span is a multiple of 64, so whole wavefronts take this branch
        if (i < span) {
#pragma unroll
            for (int s = 0; s < NDIR; ++s) {
                const uint64_t word = __ballot(arrived[s]);
                if ((threadIdx.x & 63) == 0) words[s][i >> 6] = word;
            }
        }
    };
    // the first part outside the loop, so that nothing waits for the loads
    // issued before the call
    part(0);
    for (int base = NT; base < span; base += NT) part(base);
    __syncthreads();
}

__device__ __forceinline__ int popcount_words(const uint64_t* words, int nw) {
    int c = 0;
    for (int w = 0; w < nw; ++w) c += __popcll(uniform64(words[w]));
    return c;
}

// ---------------------------------------------------------------------------
// Tiles of the per-packet kernels: a workgroup of NT threads owns a chunk of
// NT * 8 elements of one packet, thread t elements e0 .. e0 + nv - 1.
// ---------------------------------------------------------------------------
struct Chunk {
    int64_t k;    // packet
    int c;        // chunk within the packet
    int64_t c0;   // first element of the chunk
    int cv;       // valid elements of the chunk (0 .. NT * 8)
    int64_t e0;   // first element of this thread
    int lane;     // e0 - c0
    int nv;       // valid elements of this thread (0..8)
    bool whole;   // wave-uniform: every thread owns 0 or 8 elements, 16-byte aligned
};

// Chunk of tile b (tile = packet * cpp + chunk within the packet).  A chunk
// is whole when it starts on a multiple of 8 elements and its valid part
// ends on one or fills it: then every access of the tile can be a 16-byte
// vector (row starts are 16-byte aligned).
template <int NT>
__device__ __forceinline__ Chunk chunk_at(int64_t b, int64_t d, int64_t L, int cpp) {
    Chunk ch;
    ch.k = b / cpp;
    ch.c = (int)(b - ch.k * cpp);
    const int64_t pk0 = ch.k * L;
    const int64_t pend = pk0 + L < d ? pk0 + L : d;
    ch.c0 = pk0 + (int64_t)ch.c * (NT * kElems);
    const int64_t cv = pend - ch.c0;
    ch.cv = cv <= 0 ? 0 : (cv >= NT * kElems ? NT * kElems : (int)cv);
    ch.lane = (int)threadIdx.x * kElems;
    ch.e0 = ch.c0 + ch.lane;
    const int64_t rem = pend - ch.e0;
    ch.nv = rem <= 0 ? 0 : (rem >= 8 ? 8 : (int)rem);
    ch.whole = (ch.c0 % 8 == 0) && ((pend - ch.c0) % 8 == 0 || pend >= ch.c0 + NT * kElems);
    return ch;
}

// Accesses of a thread's 8 elements of the chunk of a contiguous array or
// row (`base` points at its element 0).  Whole tiles (W) go through a buffer
// resource holding the chunk's valid bytes: its base is the same for every
// lane, each lane adds a 32-bit offset, and lanes past the data read zeros
// and write nothing.  Other tiles take the element-by-element form.
template <class T>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t chunk_rsrc(const T* base, const Chunk& ch) {
    return row_rsrc(base + ch.c0, ch.cv * (int)sizeof(T));
}

template <bool W>
__device__ __forceinline__ void load_chunk(const float* base, const Chunk& ch, Raw8<F32>& r) {
    if (W) load_buf(chunk_rsrc(base, ch), ch.lane * 4, r);
    else load_raw<false>(base + ch.e0, ch.nv, r);
}

// Plain (temporal) stores: master and moments are read again next step.
template <bool W>
__device__ __forceinline__ void store_chunk(float* base, const Chunk& ch, const float (&x)[8]) {
    if (W) {
        const __amdgpu_buffer_rsrc_t r = chunk_rsrc(base, ch);
        const u32x4 a = {__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]),
                         __float_as_uint(x[3])};
        const u32x4 b = {__float_as_uint(x[4]), __float_as_uint(x[5]), __float_as_uint(x[6]),
                         __float_as_uint(x[7])};
        __builtin_amdgcn_raw_buffer_store_b128(a, r, ch.lane * 4, 0, 0);
        __builtin_amdgcn_raw_buffer_store_b128(b, r, ch.lane * 4 + 16, 0, 0);
    } else {
        store_f32x8<false>(base + ch.e0, ch.nv, x);
    }
}

// Cache-policy bit of a non-temporal buffer store (gfx940-family `nt`).
constexpr int kBufferNonTemporal = 2;

// Replica rows: non-temporal stores of the rounded values.
template <bool W>
__device__ __forceinline__ void store_chunk(float* row, const Chunk& ch, const Packed8<F32>& x) {
    if (W) {
        const __amdgpu_buffer_rsrc_t r = chunk_rsrc(row, ch);
        __builtin_amdgcn_raw_buffer_store_b128(x.r.a, r, ch.lane * 4, 0, kBufferNonTemporal);
        __builtin_amdgcn_raw_buffer_store_b128(x.r.b, r, ch.lane * 4 + 16, 0, kBufferNonTemporal);
    } else {
        x.template store<false>(row + ch.e0, ch.nv);
    }
}

template <bool W>
__device__ __forceinline__ void store_chunk(uint16_t* row, const Chunk& ch,
                                            const Packed8<BF16>& x) {
    if (W)
        __builtin_amdgcn_raw_buffer_store_b128(x.r.a, chunk_rsrc(row, ch), ch.lane * 2, 0,
                                               kBufferNonTemporal);
    else
        x.template store<false>(row + ch.e0, ch.nv);
}

// ---------------------------------------------------------------------------
// Streaming the rows of a packet chunk.
// ---------------------------------------------------------------------------
// Ascending walk over the rows whose bit is set in mask words (LDS,
// wave-uniform) or, with `invert`, clear; row `skip` (or -1) is left out.
// next() gives -1 after the last row.
struct RowWalk {
    const uint64_t* words;
    int n, nw, w, skip;
    bool invert;
    uint64_t bits;
    __device__ __forceinline__ uint64_t word(int i) const {
        uint64_t x = uniform64(words[i]);
        if (invert) x = ~x;
        const int last = n - i * 64;
        if (last < 64) x &= (1ull << last) - 1;
        if (skip >= 0 && (skip >> 6) == i) x &= ~(1ull << (skip & 63));
        return x;
    }
    __device__ __forceinline__ RowWalk(const uint64_t* words_, int n_, bool invert_, int skip_)
        : words(words_), n(n_), nw((n_ + 63) >> 6), w(0), skip(skip_), invert(invert_) {
        bits = nw > 0 ? word(0) : 0ull;
    }
    __device__ __forceinline__ int next() {
        while (bits == 0) {
            if (w + 1 >= nw) return -1;
            bits = word(++w);
        }
        const int r = w * 64 + __builtin_ctzll(bits);
        bits &= bits - 1;
        return r;
    }
};

// Hands the rows that `walk` yields, in ascending order, to use(raw) with D
// row loads in flight per thread: the load of the row D places further on is
// issued, after pace(row), as soon as a row has been used.  Whole tiles (W)
// load through buffer resources; past the last row the ring issues loads of
// size 0.  Every turn of the ring issues the same D loads and the loop is left
// only at the end of a turn, so the compiler waits for exactly one row before
// each use.
template <int D, class E, bool W, class PaceFn, class UseFn>
__device__ __forceinline__ void stream_rows(const typename E::T* rows, int64_t ld,
                                            const Chunk& ch, RowWalk& walk, const PaceFn& pace,
                                            const UseFn& use) {
    const int lane = (int)threadIdx.x * kElems * (int)sizeof(typename E::T);
    const int bytes = ch.cv * (int)sizeof(typename E::T);
    int r[D];
    Raw8<E> b[D];
#pragma unroll
    for (int u = 0; u < D; ++u) r[u] = walk.next();
    if (r[0] < 0) return;
    const int first = r[0];
    auto issue = [&](int row, Raw8<E>& x) {
        const int at = __builtin_amdgcn_readfirstlane(row >= 0 ? row : first);
        if (W) {
            load_buf(row_rsrc(rows + (int64_t)at * ld + ch.c0, row >= 0 ? bytes : 0), lane, x);
        } else {
            load_raw<false>(rows + (int64_t)at * ld + ch.e0, ch.nv, x);
        }
    };
#pragma unroll
    for (int u = 0; u < D; ++u) {
        if (r[u] >= 0) pace(r[u]);
        issue(r[u], b[u]);
    }
    for (;;) {
#pragma unroll
        for (int u = 0; u < D; ++u) {
            if (r[u] >= 0) {
                use(b[u]);
                r[u] = walk.next();
                if (r[u] >= 0) pace(r[u]);
            }
            issue(r[u], b[u]);
        }
        // rows are ascending: no row issued in this turn means every row is used
        if (r[0] < 0) return;
    }
}

// ---------------------------------------------------------------------------
// Row pacing.  Workgroups that stream many rows at the same column offset
// reach the HBM much faster when all of them touch the same row at the same
// time (a few concurrent row streams instead of one per row).  A paced kernel
// therefore issues the access of row i of a phase no earlier than a slot time
// read from the constant-rate 100 MHz clock that every compute unit sees; the
// schedule only delays accesses, so results never depend on it.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t clock_ticks() { return __builtin_amdgcn_s_memrealtime(); }

// Accessors without pacing (one-stage kernels and the unpaced fused step).
struct NoPace {
    __device__ __forceinline__ void fetch() const {}
    __device__ __forceinline__ void begin() {}
    __device__ __forceinline__ void grad(int) const {}
    __device__ __forceinline__ void rep(int) const {}
    __device__ __forceinline__ void stale(int) const {}
};

// Slot times of one round of a paced kernel, in 1/256 clock ticks: the
// access of row i in the gradient, replica and stale-read sweeps waits for
// base + off + i * delta of that sweep.  A slot further away than `guard`
// ticks (a stale or foreign anchor) is not waited for, so every wait ends.
struct ClockPace;

// Rows in flight per thread of each sweep, by pacing.  Paced, the whole chip
// streams each row at its slot, and two rows in flight keep the sweeps at the
// schedule's rate while queueing half as much in the memory system as four:
// with four, a memory stall left more workgroups late and far more steps
// slipped (the 7B-shard step kept its schedule in 7-71% of steps with four,
// 71-97% with two, on the same three boxes).
template <class Pace>
struct RingDepth {
    static constexpr int grad = kDepthGrad, stale = kDepthStale;
};
template <>
struct RingDepth<ClockPace> {
    static constexpr int grad = 2, stale = 2;
};

struct ClockPace {
    uint64_t base;  // round start, ticks (set by begin())
    uint64_t off_g, off_r, off_s;  // sweep starts, 1/256 ticks after base
    uint64_t dg, dr, ds;           // slot lengths, 1/256 ticks
    uint64_t guard;                // ticks
    // Inputs of begin(): the schedule's anchor (read by fetch() into LDS
    // before a barrier that precedes begin()) and this round's start after it.
    const uint64_t* anchor_src;
    uint64_t* anchor;  // LDS
    uint64_t round_start;
    __device__ __forceinline__ void fetch() const {
        if (threadIdx.x == 0)
            *anchor = __hip_atomic_load(anchor_src, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // Every workgroup keeps its round's slots: one that starts late issues the
    // rows whose slots have passed at once and then follows the schedule.
    // Called after the tile's first loads are issued, so the anchor's load
    // overlaps them.
    __device__ __forceinline__ void begin() { base = *anchor + round_start; }
    __device__ __forceinline__ void at(uint64_t off, uint64_t delta, int i) const {
        const uint64_t t = base + ((off + (uint64_t)i * delta) >> 8);
        uint64_t now = clock_ticks();
        if (t <= now || t - now > guard) return;
        // every waiting wave reads the shared clock; far from the slot it
        // sleeps longer between reads (s_sleep n: about 64 n core clocks,
        // 27 n ns at 2.4 GHz, so no sleep overshoots the slot)
        while (now < t) {
            const uint64_t rem = t - now;
            if (rem > 100) __builtin_amdgcn_s_sleep(16);
            else if (rem > 20) __builtin_amdgcn_s_sleep(4);
            else __builtin_amdgcn_s_sleep(1);
            now = clock_ticks();
        }
    }
    __device__ __forceinline__ void grad(int i) const { at(off_g, dg, i); }
    __device__ __forceinline__ void rep(int i) const { at(off_r, dr, i); }
    __device__ __forceinline__ void stale(int i) const { at(off_s, ds, i); }
};

// ---------------------------------------------------------------------------
// Aggregate of one packet's contributions, 8 elements per thread.
// ---------------------------------------------------------------------------
enum { kEstArrivedMean = 0, kEstHorvitzThompson = 1, kEstStaleFill = 2 };

struct AggVariant {
    int kind;                 // kEst*
    int owner;                // row that cannot be lost, or -1
    float invq;               // 1 / arrival probability (Horvitz-Thompson)
    const uint8_t* reliable;  // [P] packets that cannot be lost, or null
    void* g_prev;             // [n][ld] last arrived contributions (stale fill)
    // Horvitz-Thompson under parity packets with the arrival probability
    // derived per packet: group size (0 = use invq as given) and q.
    int parity_group;
    double q;
    // Horvitz-Thompson under Gilbert-Elliott loss with the arrival
    // probability derived per packet from the chain (ge_derived != 0).
    int ge_derived;
    double p_gb, p_bg, loss_good, loss_bad;
};

// 1 / marginal arrival probability of packet k of step t under the
// Gilbert-Elliott chain: started in Good before step 0 and moved once before
// each packet, it has made n = t P + k + 1 moves, so P(Bad) = pi_B (1 -
// (1 - p_gb - p_bg)^n) with pi_B = p_gb / (p_gb + p_bg).
__device__ __forceinline__ float ge_invq(const AggVariant& v, uint64_t t, int64_t k, int64_t P) {
    const double n = (double)t * (double)P + (double)k + 1.0;
    const double s = v.p_gb + v.p_bg;
    const double bad = s == 0.0 ? 0.0 : (v.p_gb / s) * (1.0 - pow(1.0 - s, n));
    const double q = 1.0 - (bad * v.loss_bad + (1.0 - bad) * v.loss_good);
    return (float)(1.0 / q);
}

// 1 / arrival probability of lossy packet k (of P) of a row under parity
// packets: it arrives, or it alone was lost in its group of g packets (the
// last group may be shorter) while the g - 1 - r other lossy members (r =
// reliable others) and the group's parity packet arrived: q + (1 - q) q^(g - r).
__device__ __forceinline__ float parity_invq(const AggVariant& v, int64_t k, int64_t P) {
    const int64_t g0 = (k / v.parity_group) * v.parity_group;
    const int64_t g1 = g0 + v.parity_group < P ? g0 + v.parity_group : P;
    int r = 0;
    if (v.reliable)
        for (int64_t j = g0; j < g1; ++j) r += (j != k && v.reliable[j] != 0) ? 1 : 0;
    double qn = 1.0;
    for (int64_t e = 0; e < g1 - g0 - r; ++e) qn *= v.q;
    return (float)(1.0 / (v.q + (1.0 - v.q) * qn));
}

// Arrived mean (Section 3 step (2)): g = (sum over arrived rows, ascending, in
// fp32) / K, or lam * theta when K = 0.
// Horvitz-Thompson: g = (sum over arrived lossy rows * (1/q) + the owner's row)
// / n; on a reliable packet every row has weight 1, g = sum / n.
// Stale fill (Algorithm 1): every row in ascending order contributes its
// arrived value or, if lost, its last arrived one from g_prev; arrived values
// are written to g_prev; g = sum / n.
template <class E, bool W, class Pace>
__device__ __forceinline__ void aggregate8(const typename E::T* grads, int64_t ld, const Chunk& ch,
                                           const uint64_t* gm, int n, int K, float lam,
                                           const float (&th)[8], const AggVariant& var,
                                           bool reliable_packet, const Pace& pace,
                                           float (&g)[8]) {
    const int64_t e0 = ch.e0;
    const int nv = ch.nv;
#pragma unroll
    for (int j = 0; j < 8; ++j) g[j] = 0.0f;
    if (var.kind == kEstStaleFill) {
        typename E::T* prev = reinterpret_cast<typename E::T*>(var.g_prev);
        for (int i0 = 0; i0 < n; i0 += kBatchGrad) {
            Raw8<E> raw[kBatchGrad];
            bool arr[kBatchGrad];
#pragma unroll
            for (int u = 0; u < kBatchGrad; ++u) {
                const int row = i0 + u < n ? i0 + u : i0;
                arr[u] = (uniform64(gm[row >> 6]) >> (row & 63)) & 1;
                const typename E::T* src = arr[u] ? grads : prev;
                pace.grad(row);
                load_raw<W>(src + (int64_t)row * ld + e0, nv, raw[u]);
            }
#pragma unroll
            for (int u = 0; u < kBatchGrad; ++u) {
                if (i0 + u < n) {
                    float x[8];
                    unpack(raw[u], x);
#pragma unroll
                    for (int j = 0; j < 8; ++j) g[j] += x[j];
                    if (arr[u]) store_raw<W>(prev + (int64_t)(i0 + u) * ld + e0, nv, raw[u]);
                }
            }
        }
        const float nf = (float)n;
#pragma unroll
        for (int j = 0; j < 8; ++j) g[j] = g[j] / nf;
        return;
    }
    const bool ht = var.kind == kEstHorvitzThompson;
    const int sure_row = (ht && !reliable_packet) ? var.owner : -1;
    RowWalk walk(gm, n, false, sure_row);
    stream_rows<RingDepth<Pace>::grad, E, W>(
        grads, ld, ch, walk, [&](int row) { pace.grad(row); },
        [&](const Raw8<E>& raw) {
            float x[8];
            unpack(raw, x);
#pragma unroll
            for (int j = 0; j < 8; ++j) g[j] += x[j];
        });
    if (ht) {
        const float nf = (float)n;
        if (reliable_packet) {
#pragma unroll
            for (int j = 0; j < 8; ++j) g[j] = g[j] / nf;
        } else {
            float own[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            if (sure_row >= 0) {
                pace.grad(sure_row);
                load8<E, W>(grads + (int64_t)sure_row * ld + e0, nv, own);
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) g[j] = (g[j] * var.invq + own[j]) / nf;
        }
    } else if (K > 0) {
        const float kf = (float)K;
#pragma unroll
        for (int j = 0; j < 8; ++j) g[j] = g[j] / kf;
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) g[j] = lam * th[j];
    }
}

// ---------------------------------------------------------------------------
// Owner update (Section 3 step (3)), 8 elements, fp32.
// ---------------------------------------------------------------------------
struct OptParams {
    int kind;  // 0 SGD, 1 momentum, 2 Adam
    float lr, momentum, beta1, beta2, eps;
    float bc1, bc2;  // 1 - beta^(t+1), rounded to fp32 on the host
};

__device__ __forceinline__ void update8(const OptParams& o, float (&th)[8], float (&m)[8],
                                        float (&v)[8], const float (&g)[8]) {
    if (o.kind == 0) {
#pragma unroll
        for (int j = 0; j < 8; ++j) th[j] = th[j] - o.lr * g[j];
    } else if (o.kind == 1) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            m[j] = o.momentum * m[j] + g[j];
            th[j] = th[j] - o.lr * m[j];
        }
    } else {
        const float a1 = 1.0f - o.beta1, a2 = 1.0f - o.beta2;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            m[j] = o.beta1 * m[j] + a1 * g[j];
            v[j] = o.beta2 * v[j] + a2 * (g[j] * g[j]);
            const float mh = m[j] / o.bc1;
            const float vh = v[j] / o.bc2;
            th[j] = th[j] - o.lr * (mh / (sqrtf(vh) + o.eps));
        }
    }
}

// ---------------------------------------------------------------------------
// Drift accumulation for the 8 elements of one thread.  Values are compared
// with the reference r = c(theta) of the element: d = x - r in fp64.
// ---------------------------------------------------------------------------
// Range bounds of one thread's 8 elements: the largest and smallest value
// seen per element, as floats.
struct FloatBounds8 {
    float hi[8], lo[8];
    __device__ __forceinline__ void init(int j, float h, float l) {
        hi[j] = h;
        lo[j] = l;
    }
    __device__ __forceinline__ void add(int j, float x) {
        hi[j] = fmaxf(hi[j], x);
        lo[j] = fminf(lo[j], x);
    }
    __device__ __forceinline__ float high(int j) const { return hi[j]; }
    __device__ __forceinline__ float low(int j) const { return lo[j]; }
};

// The same for values that are bf16 (rows of bf16 replicas): kept as bf16
// bit patterns, two to a register, so nothing is rounded.  Half the
// registers of FloatBounds8 for a few more ALU operations per value; the
// fused step, whose occupancy is set by its registers and which reads only
// the stale rows, takes this form; the standalone drift pass, which reads
// every row, keeps FloatBounds8.
struct Bf16Bounds8 {
    uint32_t hi[4], lo[4];
    __device__ __forceinline__ static float get(const uint32_t (&w)[4], int j) {
        return __uint_as_float((j & 1) ? (w[j >> 1] & 0xFFFF0000u) : (w[j >> 1] << 16));
    }
    __device__ __forceinline__ static void put(uint32_t (&w)[4], int j, float v) {
        const uint32_t b = __float_as_uint(v) >> 16;
        w[j >> 1] = (j & 1) ? ((w[j >> 1] & 0xFFFFu) | (b << 16)) : ((w[j >> 1] & 0xFFFF0000u) | b);
    }
    __device__ __forceinline__ void init(int j, float h, float l) {
        put(hi, j, h);
        put(lo, j, l);
    }
    __device__ __forceinline__ void add(int j, float x) {
        put(hi, j, fmaxf(get(hi, j), x));
        put(lo, j, fminf(get(lo, j), x));
    }
    __device__ __forceinline__ float high(int j) const { return get(hi, j); }
    __device__ __forceinline__ float low(int j) const { return get(lo, j); }
};

template <class R>
struct StepBounds8 {
    using type = FloatBounds8;
};
template <>
struct StepBounds8<BF16> {
    using type = Bf16Bounds8;
};

template <class B>
struct Drift8 {
    double s1[8], s2[8];
    B b;
    double abs_sum;

    __device__ __forceinline__ void init(bool any_equal_ref, const float (&r)[8]) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            s1[j] = 0.0;
            s2[j] = 0.0;
            b.init(j, any_equal_ref ? r[j] : -__builtin_inff(),
                   any_equal_ref ? r[j] : __builtin_inff());
        }
        abs_sum = 0.0;
    }
    __device__ __forceinline__ void add(const float (&x)[8], const float (&r)[8], int nv) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (j < nv) {
                const double d = (double)x[j] - (double)r[j];
                s1[j] = s1[j] + d;
                s2[j] = __fma_rn(d, d, s2[j]);
                abs_sum = abs_sum + fabs(d);
                b.add(j, x[j]);
            }
        }
    }
    // Fold into per-thread totals: pair sum N*S2 - S1^2 per element (clamped
    // at 0 against rounding, so that identical rows give exactly 0) and the
    // max range.
    __device__ __forceinline__ void finish(int n, int nv, double& pair, double& range) const {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (j < nv) {
                const double ps = (double)n * s2[j] - s1[j] * s1[j];
                pair = pair + (ps > 0.0 ? ps : 0.0);
                const double rg = (double)b.high(j) - (double)b.low(j);
                range = rg > range ? rg : range;
            }
        }
    }
};

struct DriftPartial {
    double pair, abs_sum, range;
    uint32_t stale, empty;
};

// Fixed-order reduction of (pair, abs, range) over a workgroup of NT
// threads; thread 0 writes the partial with the packet bookkeeping counts.
template <int NT>
__device__ __forceinline__ void block_reduce_partial(double pair, double abs_sum,
                                                     double range, uint32_t stale,
                                                     uint32_t empty, DriftPartial* out) {
    __shared__ double s_red[3][NT / 64];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        pair += __shfl_down(pair, off, 64);
        abs_sum += __shfl_down(abs_sum, off, 64);
        const double r2 = __shfl_down(range, off, 64);
        range = r2 > range ? r2 : range;
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        s_red[0][wave] = pair;
        s_red[1][wave] = abs_sum;
        s_red[2][wave] = range;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double p = 0.0, a = 0.0, r = 0.0;
        for (int w = 0; w < NT / 64; ++w) {
            p += s_red[0][w];
            a += s_red[1][w];
            r = s_red[2][w] > r ? s_red[2][w] : r;
        }
        DriftPartial dp;
        dp.pair = p;
        dp.abs_sum = a;
        dp.range = r;
        dp.stale = stale;
        dp.empty = empty;
        *out = dp;
    }
}

}  // namespace lossy
