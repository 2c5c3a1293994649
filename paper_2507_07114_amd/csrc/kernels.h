// Internal interface between the C ABI (api.cpp) and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lossy_device.h"

namespace lossy {

// Mirror of ll_drift (device-written).
struct DriftOut {
    double max_abs, mean_sq, rms, mean_abs_to_master;
    unsigned long long stale_packets, empty_packets;
};

// Running totals of drift partials (second reduction level), 64-bit counts.
struct DriftAcc {
    double pair, abs_sum, range;
    unsigned long long stale, empty;
    __device__ __forceinline__ void zero() {
        pair = abs_sum = range = 0.0;
        stale = empty = 0;
    }
    __device__ __forceinline__ void add(const DriftPartial& q) {
        pair += q.pair;
        abs_sum += q.abs_sum;
        range = q.range > range ? q.range : range;
        stale += q.stale;
        empty += q.empty;
    }
    __device__ __forceinline__ void add(const DriftAcc& q) {
        pair += q.pair;
        abs_sum += q.abs_sum;
        range = q.range > range ? q.range : range;
        stale += q.stale;
        empty += q.empty;
    }
};

struct GeParams {
    uint64_t seed;
    uint64_t thr_gb, thr_bg, thr_loss_good, thr_loss_bad;
};

// Workgroups of the first drift reduction level.
constexpr int kReduceGroups = 256;

// The second-level partials are followed by the counter with which the last
// reducing workgroup finds itself.
__host__ __device__ inline unsigned* reduce_counter(DriftAcc* groups) {
    return reinterpret_cast<unsigned*>(groups + kReduceGroups);
}
constexpr size_t kReduceBytes = kReduceGroups * sizeof(DriftAcc) + 16;

// Gilbert-Elliott scan geometry: a thread composes kGeRun consecutive packets,
// a workgroup one segment of kGeSeg packets.
constexpr int kGeRun = 16;
constexpr int64_t kGeSeg = (int64_t)kThreads * kGeRun;

// One direction's Gilbert-Elliott chains (scratch regions from the workspace).
struct GeJob {
    GeParams ge;
    uint64_t dir;
    uint8_t* state;     // [n] chain state, in/out
    uint8_t* arrived;   // [n][P] out
    uint8_t* tmaps;     // [n][S][kThreads] per-run composite maps (scratch)
    uint8_t* comps;     // [n][S] per-segment composite maps (scratch)
    uint8_t* state_in;  // [n] copy of the input state (scratch)
    int owner;                // row that always arrives, or -1
    const uint8_t* reliable;  // [P] packets that always arrive, or null
};

struct GeLaunch {
    int n;
    int64_t P, S;  // packets, segments of kGeSeg packets
    uint64_t step;
    GeJob job[2];
};

struct AggParams {
    int n;
    int64_t d, L, P;
    int cpp;  // chunks per packet (set by the launcher)
    const void* grads;
    int64_t ld;
    const uint8_t* arrived;
    float lam;
    const float* theta;
    float* g_hat;
    int32_t* counts;
    AggVariant var;
};

struct BcastParams {
    int n;
    int64_t d, L, P;
    int cpp;
    const float* theta;
    void* replicas;
    int64_t ld;
    const uint8_t* arrived;
};

struct DriftParams {
    int n;
    int64_t d, L, P;
    int cpp;
    const void* replicas;
    int64_t ld;
    const float* theta;
    const uint8_t* arrived;
    DriftPartial* partials;
    DriftAcc* groups;  // [kReduceGroups] second-level partials, then the counter
};

struct FusedParams {
    int n;
    int64_t d, L, P;
    int cpp;
    uint64_t step;
    MaskSource src[2];  // [0] gradient, [1] broadcast
    uint8_t* out_g;
    uint8_t* out_b;
    int32_t* counts;
    const void* grads;
    int64_t ld_g;
    OptParams opt;
    float lam;
    float* theta;
    float* m;
    float* v;
    void* replicas;
    int64_t ld_r;
    DriftPartial* partials;
    DriftAcc* groups;  // [kReduceGroups] second-level partials, then the counter
    AggVariant var;
    uint16_t* ages;    // [n][P] broadcast ages, or null
    // [n][P] memory where a paced step may draw each direction's Bernoulli
    // masks beforehand (the caller's mask output or workspace), or null.
    uint8_t* pre[2];
};

// Slot schedule of the paced fused step (see ClockPace), times in 1/256
// clock ticks relative to each round's start.
struct PaceParams {
    int64_t per_round;             // workgroups (tiles) per round
    uint64_t round;                // time between round starts
    uint64_t off_g, off_r, off_s;  // gradient, replica and stale-read sweep starts
    uint64_t dg, dr, ds;           // slot lengths of the three sweeps
    uint64_t guard;                // longest wait, ticks
};

// Pacing modes and defaults: auto paces steps of at least kPaceMinRows rows
// spanning at least kPaceMinRounds rounds (of at most kPaceMaxRoundTiles
// tiles for fp32 rows); the schedule is laid out for kDefaultPaceRate bytes/s
// (kDefaultPaceRateF32 for steps with fp32 replica rows) with
// kDefaultPaceGapUs between the gradient and replica sweeps, and starts
// kPaceMarginUs after the anchor is written.
enum { kPaceAuto = 0, kPaceAlways = 1, kPaceNever = 2 };
constexpr int64_t kPaceMinRounds = 8;
constexpr int kPaceMinRows = 32;
constexpr int64_t kPaceMaxRoundTiles = 1024;
constexpr double kDefaultPaceRate = 6.3e12;
constexpr double kDefaultPaceRateF32 = 5.9e12;
constexpr double kDefaultPaceGapUs = 2.0;
constexpr double kDefaultPaceLeadUs = 4.0;
constexpr int kDefaultPaceOverlap = 1;
constexpr int kDefaultPaceResident = 1;
constexpr double kPaceMarginUs = 3.0;
constexpr double kDefaultPaceTailUs = 3.0;
constexpr int kDefaultPacePersistent = 0;
// Fraction of the resident workgroup places the rounds in flight may fill.
constexpr double kDefaultPaceHeadroom = 1.0;

// How the fused step is paced (process-wide; see ll_set_pacing).
struct PaceSetting {
    int mode;            // 0 auto, 1 always, 2 never
    double bytes_per_s;  // rate the schedule is laid out for
    double gap_us;       // allowance between the last gradient row and the first replica row
    double lead_us;      // allowance from a round's start to its first gradient row
    int overlap;         // rounds streaming at once (1 or 2)
    int resident;        // rounds the resident workgroup places are shared by (>= overlap)
    double headroom;     // fraction of the resident places the rounds may fill
    double tail_us;      // allowance after a round's last slot
    int persistent;      // 1: one round of workgroups loops over the rounds (plain steps)
    double bytes_per_s_f32;  // rate for steps whose replica rows are fp32
};
PaceSetting get_pace_setting();
void set_pace_setting(const PaceSetting& s);

// Expected arrival probabilities of a step, for laying out its schedule.
struct PaceHint {
    double q_g, q_b;
};

// Largest packet group of the parity-packet recovery.
constexpr int kMaxParityGroup = 256;

// One direction's Bernoulli masks (with parity recovery in k_masks_parity).
struct MaskJob {
    uint64_t dir, seed, thr;
    int owner;
    const uint8_t* reliable;  // [P] or null
    uint8_t* arrived;         // [n][P] out
};

// A workgroup covers `span` consecutive packets of one row, span = G *
// floor(kThreads / G), so groups never straddle workgroups.
struct ParityLaunch {
    int ndir, n, G, span;
    int64_t P, spans;  // spans = ceil(P / span) per row
    uint64_t step;
    MaskJob job[2];
};

hipError_t launch_masks_parity(const ParityLaunch& L, hipStream_t s);
hipError_t launch_masks_bernoulli_jobs(int n, int64_t num_packets, uint64_t step,
                                       const MaskJob* jobs, int njobs, hipStream_t s);
hipError_t launch_masks_bernoulli(int n, int64_t num_packets, uint64_t step, int dir,
                                  uint64_t seed, uint64_t thr, int owner,
                                  const uint8_t* reliable, uint8_t* arrived, hipStream_t s);
hipError_t launch_ages_update(int64_t total, const uint8_t* arrived, uint16_t* ages,
                              hipStream_t s);
hipError_t launch_masks_ge(const GeLaunch& L, int ndir, hipStream_t s);
hipError_t launch_aggregate(int gdtype, const AggParams& p, hipStream_t s);
hipError_t launch_shard_step(int64_t d, const OptParams& o, float* theta, float* m, float* v,
                             const float* g_hat, hipStream_t s);
hipError_t launch_broadcast(int rdtype, const BcastParams& p, hipStream_t s);
hipError_t launch_drift(int rdtype, const DriftParams& p, int n, int64_t d, int have_master,
                        DriftOut* out, hipStream_t s);
hipError_t launch_fused(int gdtype, int rdtype, const FusedParams& p, DriftOut* drift,
                        const PaceHint& hint, hipStream_t s);
hipError_t launch_drift_zero(DriftOut* out, hipStream_t s);

// Device scratch of the entry point that allocates nothing: a static device
// array of kNoAllocScratchBytes per device.  noalloc_scratch gives its
// address on the current device (looked up once per device, at most
// kMaxDevices devices).
constexpr size_t kNoAllocScratchBytes = (size_t)16 << 20;
constexpr int kMaxDevices = 64;
hipError_t noalloc_scratch(void** ptr);

}  // namespace lossy
