/*
 * lossy.h -- C ABI of the packet-loss-tolerant data-parallel step on one
 * MI355X (gfx950).
 *
 * The operations follow "Distributed Training under Packet Loss"
 * (Weintraub, Banner, Orda, 2025), Section 3, for the shard owned by one
 * worker W_j.  N workers each hold a gradient row for that shard; the shard
 * of D elements is cut into packets of L elements (P = ceil(D / L) packets,
 * the last may be short).  Per step:
 *
 *   (a) gradient packets from each worker arrive or are lost (step (2));
 *   (b) the owner forms the unbiased aggregate: per packet, the sum of the
 *       rows that arrived divided by how many arrived (step (2) and
 *       "Unbiased Gradient Aggregation");
 *   (c) the owner updates its fp32 master shard (step (3));
 *   (d) the owner broadcasts the new shard; each of the N replica buffers
 *       takes a packet only where that broadcast arrived, otherwise keeps
 *       its stale value (step (4));
 *   (e) drift statistics over the N replicas (Theorem 3.1).
 *
 * Conventions for every entry point:
 *   - All pointers are DEVICE pointers unless marked "host".  The caller owns
 *     all memory; the library allocates none.  Scratch memory comes from a
 *     caller-supplied workspace of ll_workspace_bytes() bytes (or, for
 *     lossy_step_fused_noalloc, from a static device array of the library).
 *   - `stream` is a hipStream_t (NULL = the default stream).  Every call only
 *     enqueues kernels on it (no allocation, no memset, no copy) and returns
 *     without synchronising; device outputs are valid once the stream has
 *     reached that point.  Calls can therefore be captured into a HIP graph;
 *     a replay repeats the captured step index.
 *   - Row-major [N][ld] buffers: row i starts at element i * ld.  ld >= D and
 *     ld times the element size (4 bytes fp32, 2 bytes bf16) is a multiple of
 *     16 bytes, so every row starts on a 16-byte boundary.
 *   - Any packet length L >= 1 is accepted.  Packets whose start is a multiple
 *     of 8 elements (L a multiple of 8) are moved with 16-byte vector accesses;
 *     other packets, and the last 1..7 elements of a shard whose D is not a
 *     multiple of 8, are moved element by element (same results, slower).
 *   - Masks are uint8 [N][P] (row i = worker/replica i, column k = packet),
 *     1 = arrived, 0 = lost.
 *   - Return codes: LL_OK (0); LL_EINVAL (-1) for a bad size or argument
 *     (N outside [1, 1024], D < 0, L < 1, ld < D,
 *     a probability outside [0, 1], an unknown kind or dtype, a required
 *     pointer that is NULL, a workspace that is too small, or a launch that
 *     would exceed the grid limit); LL_EALIGN (-2) when a buffer address is
 *     not 16-byte aligned or ld * element size is not a multiple of 16; LL_EHIP
 *     (-3) when the HIP runtime reports an error.  ll_last_error() then
 *     returns a message (thread-local, valid until the next call on that
 *     thread).  No exception crosses this boundary.
 *   - D = 0 is a valid no-op (drift outputs are then written as zeros).
 *   - Calls that share output buffers must be ordered by the caller (same
 *     stream or events); the library keeps no state between calls.
 */
#ifndef LOSSY_H
#define LOSSY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define LL_API __attribute__((visibility("default")))
#else
#define LL_API
#endif

enum { LL_OK = 0, LL_EINVAL = -1, LL_EALIGN = -2, LL_EHIP = -3 };
enum { LL_F32 = 0, LL_BF16 = 1 };
enum { LL_LOSS_BERNOULLI = 0, LL_LOSS_GILBERT_ELLIOTT = 1 };
enum { LL_SGD = 0, LL_SGD_MOMENTUM = 1, LL_ADAM = 2 };
enum { LL_DIR_GRAD = 0, LL_DIR_BCAST = 1 };
enum { LL_EST_ARRIVED_MEAN = 0, LL_EST_HORVITZ_THOMPSON = 1, LL_EST_STALE_FILL = 2 };

/*
 * Loss process (Section 3 steps (2) and (4): each transfer succeeds with
 * probability 1 - p; Algorithm 1 drops when Uniform(0,1) < p).
 *
 * The draw for step t (0-based), worker i, packet k and direction dir is the
 * Philox4x64-10 block (Salmon et al., SC'11) at counter (k, i, t, dir) under
 * key (seed, 0).  With u0, u1 the top 32 bits of its words 0 and 1:
 *   BERNOULLI        lost  <=>  u0 < ceil(p * 2^32)   (so u0 / 2^32 < p).
 *   GILBERT_ELLIOTT  per (dir, worker) a two-state chain over packets in
 *                    step-major order, Good before step 0; per packet the
 *                    state first moves (Good->Bad iff u0 < ceil(p_gb 2^32),
 *                    Bad->Good iff u0 < ceil(p_bg 2^32)), then the packet is
 *                    lost iff u1 < ceil(loss_state 2^32).  Bursty loss goes
 *                    beyond the paper's i.i.d. model (its Section 5).
 * Fields not used by `kind` are ignored.
 */
typedef struct {
    int32_t kind;
    double p;
    double p_gb, p_bg, loss_good, loss_bad;
    uint64_t seed;
} ll_loss;

/*
 * Owner update (Section 3 step (3): theta <- theta - eta * g_hat).
 *   LL_SGD           theta -= lr * g
 *   LL_SGD_MOMENTUM  b = momentum * b + g;  theta -= lr * b   (b starts at 0)
 *   LL_ADAM          m = beta1 m + (1-beta1) g;  v = beta2 v + (1-beta2) g^2;
 *                    theta -= lr * (m / (1-beta1^(t+1))) /
 *                             (sqrt(v / (1-beta2^(t+1))) + eps)
 * fallback_lambda: for a packet with no arrived contribution the paper
 * leaves the substitute open ("Unbiased Gradient Aggregation"); here the
 * aggregate is then fallback_lambda * theta (0 gives g_hat = 0).
 */
typedef struct {
    int32_t kind;
    float lr, momentum, beta1, beta2, eps;
    float fallback_lambda;
} ll_opt;

/*
 * Drift statistics over the N replicas x_i of every element e (the
 * discrepancy D = theta^(i,j) - theta^(k,j) of Theorem 3.1):
 *   max_abs            max_e (max_i x_ie - min_i x_ie)
 *   mean_sq            sum_e sum_{i<k} (x_ie - x_ke)^2 / (D * N(N-1)/2)
 *                      (0 when N = 1 or D = 0)
 *   rms                sqrt(mean_sq)
 *   mean_abs_to_master sum_{i,e} |x_ie - c(theta_e)| / (N D), c = rounding to
 *                      the replica dtype; NaN when no master is given
 *   stale_packets      number of (replica, packet) broadcasts lost
 *   empty_packets      packets whose gradient contributions were all lost
 *                      (filled by lossy_step_fused; drift_stats writes 0)
 * Sums are taken in fp64 in a fixed order, so results are deterministic.
 */
typedef struct {
    double max_abs, mean_sq, rms, mean_abs_to_master;
    uint64_t stale_packets, empty_packets;
} ll_drift;

/*
 * Optional variants of the step; every entry point that takes `ext` accepts
 * NULL for the defaults (all zero except owner = -1).
 *   estimator  how the owner combines a packet's contributions:
 *     LL_EST_ARRIVED_MEAN      (default) sum of the arrived contributions over
 *                              their count (Section 3 step (2)); fallback when
 *                              none arrived (see ll_opt.fallback_lambda).
 *     LL_EST_HORVITZ_THOMPSON  each arrived contribution weighted by 1/q and
 *                              the sum divided by N: unbiased with no
 *                              conditioning and no fallback.  q = arrival_prob
 *                              for lossy contributions and 1 for those that
 *                              cannot be lost (owner row, reliable packets).
 *     LL_EST_STALE_FILL        Algorithm 1's gradient half: a lost contribution
 *                              is replaced by the last one that arrived from
 *                              that worker (g_prev), an arrived one is used and
 *                              stored into g_prev; the N values are averaged.
 *   owner         -1, or the row whose gradient piece and replica stay local
 *                 (Section 3 step (4) broadcasts to the other workers): that
 *                 row always arrives, in both directions.
 *   reliable      uint8 [P] (device) or NULL: packets flagged 1 travel over a
 *                 reliable channel (the hybrid transport proposed in the
 *                 paper's Section 5) and arrive at every row, both directions.
 *   g_prev        [n][ld_g] of the gradient dtype (device, in/out), required by
 *                 LL_EST_STALE_FILL (zero before the first step), else unused.
 *   ages          uint16 [n][P] (device, in/out) or NULL; lossy_step_fused only:
 *                 steps since each replica packet last received the broadcast
 *                 (0 = this step; saturates at 65535).
 *   arrival_prob  q of LL_EST_HORVITZ_THOMPSON in (0, 1].  lossy_aggregate
 *                 requires it; lossy_step_fused takes 0 to mean each packet's
 *                 exact arrival probability under the gradient loss: q = 1 - p
 *                 for Bernoulli loss, with parity packets q + (1 - q) q^(g - r)
 *                 (g the size of the packet's group, r its reliable other
 *                 members); for Gilbert-Elliott loss the chain's marginal
 *                 1 - (b loss_bad + (1 - b) loss_good) with b = pi_B (1 -
 *                 (1 - p_gb - p_bg)^n), pi_B = p_gb / (p_gb + p_bg), after
 *                 n = step * P + k + 1 moves from Good (needs loss_good < 1 and
 *                 loss_bad < 1).
 *   parity_group  0 (none), or G in [1, 256]: erasure coding over groups of G
 *                 consecutive packets (the parity packets proposed in the
 *                 paper's Section 5).  Per row and group, the sender adds one
 *                 XOR parity packet; when exactly one packet of the group was
 *                 lost and the parity packet arrived, the receiver rebuilds
 *                 the lost packet bit for bit, so it counts as arrived.  The
 *                 last group of a row may be shorter.  The parity packet of
 *                 group j in direction dir is lost under the same Bernoulli p,
 *                 drawn with counter (j, i, t, dir + 2).  Bernoulli loss only
 *                 (LL_EINVAL for Gilbert-Elliott).  G = 1 sends every packet
 *                 twice.
 * Masks read from memory (lossy_aggregate, lossy_broadcast, drift_stats) are
 * taken as given: ll_masks and lossy_step_fused apply owner, reliable and
 * parity recovery, in that order.
 */
typedef struct {
    int32_t estimator;
    int32_t owner;
    const uint8_t* reliable;
    void* g_prev;
    uint16_t* ages;
    double arrival_prob;
    int32_t parity_group;
} ll_ext;

/*
 * Arrival masks for one step and direction (Section 3 step (2) for
 * dir = LL_DIR_GRAD, step (4) for LL_DIR_BCAST) under `loss` (host).
 *   n, num_packets   mask shape [n][num_packets]; arrived (device, out).
 *   step             0-based step index t.
 *   ge_state         Gilbert-Elliott only: uint8 [n] (device, in/out), the
 *                    chain state (0 Good, 1 Bad) at the end of the previous
 *                    step; updated to the end of this step.  Ignored (may be
 *                    NULL) for Bernoulli.
 *   workspace        Gilbert-Elliott only: device scratch of ws_bytes >=
 *                    ll_masks_workspace_bytes(n, num_packets); ignored (may be
 *                    NULL) for Bernoulli.
 *   ext              NULL, or variants: owner and reliable force arrivals;
 *                    parity_group adds parity recovery (Bernoulli only).
 */
LL_API int ll_masks(int32_t n, int64_t num_packets, uint64_t step, int32_t dir,
                    const ll_loss* loss, uint8_t* ge_state, uint8_t* arrived,
                    void* workspace, size_t ws_bytes, const ll_ext* ext, void* stream);

/* Scratch bytes ll_masks needs for a Gilbert-Elliott process (0 on invalid
 * sizes).  Bernoulli masks need none. */
LL_API size_t ll_masks_workspace_bytes(int32_t n, int64_t num_packets);

/*
 * Unbiased aggregate (Section 3 step (2); "Unbiased Gradient Aggregation"):
 *   g_hat[e] = (sum_{i : arrived[i][k(e)]} grads[i][e]) / K[k(e)],
 *   K[k] = sum_i arrived[i][k]; when K = 0, g_hat[e] = fallback_lambda * theta[e].
 * The sum runs over arrived rows in ascending i, in fp32.
 *   grads    [n][ld_g] of gdtype (LL_F32 or LL_BF16).
 *   arrived  uint8 [n][P].
 *   theta    fp32 [d]; read only when fallback_lambda != 0 (else may be NULL).
 *   g_hat    fp32 [d] (out).  counts: int32 [P] (out, may be NULL).
 *   ext      NULL, or the estimator variant (with owner and reliable naming
 *            the contributions that could not be lost, and g_prev).
 * Lost rows are never read (their g_prev is, under LL_EST_STALE_FILL).
 */
LL_API int lossy_aggregate(int32_t n, int64_t d, int64_t packet, int32_t gdtype,
                    const void* grads, int64_t ld_g, const uint8_t* arrived,
                    float fallback_lambda, const float* theta, float* g_hat,
                    int32_t* counts, const ll_ext* ext, void* stream);

/*
 * Broadcast ages (see ll_ext.ages) after a broadcast with masks arrived_bc
 * uint8 [n][num_packets]: ages[i][k] = 0 where the packet arrived, else
 * min(ages[i][k] + 1, 65535).  ages: uint16 [n][num_packets], in/out.
 */
LL_API int ll_ages_update(int32_t n, int64_t num_packets, const uint8_t* arrived_bc,
                          uint16_t* ages, void* stream);

/*
 * Owner update of the fp32 master shard (Section 3 step (3)), in place.
 *   opt (host); step = 0-based t (Adam's bias correction uses t + 1).
 *   m  momentum buffer (LL_SGD_MOMENTUM) or Adam first moment; NULL for SGD.
 *   v  Adam second moment; NULL otherwise.   g_hat fp32 [d].
 */
LL_API int shard_step(const ll_opt* opt, int64_t d, uint64_t step, float* theta,
               float* m, float* v, const float* g_hat, void* stream);

/*
 * Lossy parameter broadcast (Section 3 step (4)): for every replica i and
 * packet k with arrived_bc[i][k] = 1, replicas[i][packet k] <- c(theta)
 * (c = identity for LL_F32, round-to-nearest-even for LL_BF16); packets whose
 * broadcast was lost are neither read nor written (they keep stale values).
 *   theta fp32 [d]; replicas [n][ld_r] of rdtype; arrived_bc uint8 [n][P].
 */
LL_API int lossy_broadcast(int32_t n, int64_t d, int64_t packet, const float* theta,
                    int32_t rdtype, void* replicas, int64_t ld_r,
                    const uint8_t* arrived_bc, void* stream);

/*
 * Drift statistics (see ll_drift) over all n replicas [n][ld_r] of rdtype.
 *   theta       fp32 [d] master used as the reference c(theta); may be NULL
 *               (then replica 0 is the reference and mean_abs_to_master is NaN).
 *   arrived_bc  uint8 [n][P], only used to count stale packets; may be NULL.
 *   workspace   device scratch of ws_bytes >= ll_workspace_bytes(n, d, packet).
 *   out         ll_drift (device, out).
 */
LL_API int drift_stats(int32_t n, int64_t d, int64_t packet, int32_t rdtype,
                const void* replicas, int64_t ld_r, const float* theta,
                const uint8_t* arrived_bc, void* workspace, size_t ws_bytes,
                ll_drift* out, void* stream);

/*
 * The whole step in one pass over HBM: masks (both directions), aggregate,
 * update, broadcast and, if `drift` is non-NULL, drift statistics of the
 * replicas after the broadcast.  Equivalent to
 *   ll_masks(GRAD) -> lossy_aggregate -> shard_step -> ll_masks(BCAST)
 *   -> lossy_broadcast -> drift_stats
 * (and ll_ages_update) with the same arithmetic, so its outputs are
 * bit-identical to that chain given the same ext (except Horvitz-Thompson
 * weights derived per packet, arrival_prob = 0 under parity packets or
 * Gilbert-Elliott loss, which lossy_aggregate cannot take).
 *   loss_g, loss_b, opt     host structs.
 *   ge_state_g, ge_state_b  uint8 [n] each (device, in/out) for
 *                           Gilbert-Elliott processes, else may be NULL.
 *   arrived_g, arrived_b    uint8 [n][P] (out, may be NULL): the masks drawn.
 *   counts                  int32 [P] (out, may be NULL): gradient arrivals.
 *   workspace, ws_bytes     scratch, ws_bytes >= ll_workspace_bytes(n, d, packet);
 *                           required with drift, a Gilbert-Elliott process or
 *                           parity packets.
 *   drift                   ll_drift (device, out) or NULL to skip drift.
 *   ext                     NULL, or variants (estimator, owner, reliable,
 *                           g_prev, ages, parity_group).
 * Lost gradient packets are never read; lost broadcast packets are read only
 * for drift and never written.
 */
LL_API int lossy_step_fused(int32_t n, int64_t d, int64_t packet, uint64_t step,
                     const ll_loss* loss_g, const ll_loss* loss_b,
                     uint8_t* ge_state_g, uint8_t* ge_state_b,
                     int32_t gdtype, const void* grads, int64_t ld_g,
                     const ll_opt* opt, float* theta, float* m, float* v,
                     int32_t rdtype, void* replicas, int64_t ld_r,
                     uint8_t* arrived_g, uint8_t* arrived_b, int32_t* counts,
                     void* workspace, size_t ws_bytes, ll_drift* drift,
                     const ll_ext* ext, void* stream);

/*
 * lossy_step_fused for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops, harnesses that forbid hipMalloc):
 * the same step, arguments and results, with the workspace taken from a
 * static device array of LL_NOALLOC_SCRATCH_BYTES that the library holds on
 * every device it runs on until the process ends.  No call allocates (no
 * hipMalloc, hipFree or allocating library routine); the first call on a
 * device looks the array's address up on that device.
 *   Sizes whose workspace, ll_workspace_bytes(n, d, packet), exceeds
 *   LL_NOALLOC_SCRATCH_BYTES return LL_EINVAL before any device work.
 *   Every call on one device shares that device's array and leaves its
 *   contents behind (the step writes everything it reads from it before
 *   reading it); calls that overlap on one device (other streams, other
 *   threads) race on it and must be ordered by the caller.
 */
enum { LL_NOALLOC_SCRATCH_BYTES = 16777216 };
LL_API int lossy_step_fused_noalloc(int32_t n, int64_t d, int64_t packet, uint64_t step,
                     const ll_loss* loss_g, const ll_loss* loss_b,
                     uint8_t* ge_state_g, uint8_t* ge_state_b,
                     int32_t gdtype, const void* grads, int64_t ld_g,
                     const ll_opt* opt, float* theta, float* m, float* v,
                     int32_t rdtype, void* replicas, int64_t ld_r,
                     uint8_t* arrived_g, uint8_t* arrived_b, int32_t* counts,
                     ll_drift* drift, const ll_ext* ext, void* stream);

/*
 * Pacing of lossy_step_fused (a performance setting of this library, not part
 * of the paper's method; it never changes a result).  The fused step streams
 * all N gradient rows and all N replica rows of every packet.  When each
 * workgroup walks the rows on its own, the chip has pieces of every row in
 * flight at once and the HBM serves them well below its streaming rate.  A
 * paced step gives each workgroup one tile (a chunk of a packet, 4 KiB of
 * every row) as before, but groups the tiles into rounds of adjacent tiles;
 * in each round's sweeps (gradient rows, replica rows, stale replica rows
 * read for drift) the access of row i waits for a slot time on the 100 MHz
 * clock that all compute units share, so the chip streams a few long runs of
 * one row at a time.  A slot lasts as long as its expected bytes take at the
 * round's share of bytes_per_s; a round starts with a lead (the workgroups
 * start and read their master and moments) and has a gap between its
 * gradient and replica sweeps (the update).  Laid out too fast, the schedule
 * is not kept and the speed falls back towards the unpaced one; too slow, the
 * step runs at the set rate.
 *   mode         LL_PACE_AUTO (default): paced where it was measured to pay,
 *                steps with at least 32 workers and at least 8 rounds (few
 *                workers break even or lose); LL_PACE_ALWAYS; LL_PACE_NEVER.
 *                A round takes every resident workgroup place (bf16
 *                rows) or at most 1024 tiles (fp32 rows, 4 MiB of a row
 *                per slot).
 *   bytes_per_s  rate the slots are laid out for (default 6.3e12), for
 *                steps whose replica rows are bf16.
 *   gap_us       time between the last gradient slot and the first replica
 *                slot, besides the master and moment writes (default 2).
 *   lead_us      time from a round's start to its first gradient slot,
 *                besides the master and moment reads (default 4).
 *   overlap      rounds streaming at once (1 or 2; default 1).  With 1,
 *                rounds run back to back and the chip streams one row at a
 *                time, reading in the gradient sweep and writing in the
 *                replica sweep.  With 2, each round gets half the rate and
 *                rounds start half a round apart, so one round's gradient
 *                sweep runs beside the previous round's replica sweep and
 *                each round's lead and gap are covered by the other's
 *                streams (two mixed streams: measured to hold about 6.0e12).
 *   resident     rounds sharing the workgroup places the chip holds at once
 *                (overlap..4; default 1): a round has headroom / resident of
 *                them, and rounds start no closer than a round's length /
 *                resident apart, so that every round's workgroups find places
 *                when it starts.
 *   headroom     fraction of those places the rounds fill ((0, 1]; 1.0).
 *   tail_us      time after a round's last slot before the next round may
 *                count on its places ([0, 1e4]; default 3).
 *   persistent   1: steps in the plain configuration (arrived-mean
 *                estimator, masks drawn beforehand or from memory, no forced
 *                arrivals, ages or mask outputs beyond the drawn masks,
 *                packet length and shard a multiple of 8) run one round's
 *                worth of workgroups that loop over the rounds, so no
 *                workgroup starts or leaves between rounds; needs overlap
 *                and resident 1.  0: one workgroup per tile (default 0).
 *   bytes_per_s_f32  the same for steps whose replica rows are fp32 (their
 *                workgroups are 128 threads with two loads per row each;
 *                measured to keep their schedule at a lower rate; default
 *                5.9e12).
 * A workgroup that starts behind its round (its place freed late) issues the
 * rows whose slots have passed at once and then keeps the round's slots.
 * The setting is process-wide and read at each call.  A paced step enqueues,
 * before the step itself: the Bernoulli mask kernel for each direction whose
 * masks have memory to go to (the caller's mask output, else the workspace
 * when one of ll_workspace_bytes() bytes is passed), so that the step reads
 * its masks instead of drawing them at the start of every round; and a
 * one-lane kernel that stores the schedule's start time in a per-device
 * device variable.  Overlapping paced steps on one device can read each
 * other's start time, which costs speed but changes no result.
 * ll_set_pacing returns LL_EINVAL for an unknown mode or a field outside the
 * ranges above (bytes_per_s and bytes_per_s_f32 in (0, 1e15), gap_us,
 * lead_us and tail_us in [0, 1e4], persistent 0 or 1 and only with overlap
 * and resident 1);
 * ll_get_pacing fills `out` (host).
 */
enum { LL_PACE_AUTO = 0, LL_PACE_ALWAYS = 1, LL_PACE_NEVER = 2 };
typedef struct {
    int32_t mode;
    double bytes_per_s;
    double gap_us;
    double lead_us;
    int32_t overlap;
    int32_t resident;
    double headroom;
    double tail_us;
    int32_t persistent;
    double bytes_per_s_f32;
} ll_pacing;

LL_API int ll_set_pacing(const ll_pacing* cfg);
LL_API int ll_get_pacing(ll_pacing* out);

/* Bytes of device workspace that drift_stats and lossy_step_fused need for
 * these sizes (0 on invalid sizes): drift partials, two mask areas and the
 * Gilbert-Elliott scan scratch of both directions. */
LL_API size_t ll_workspace_bytes(int32_t n, int64_t d, int64_t packet);

/* Message describing the last error on this thread ("" if none). */
LL_API const char* ll_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LOSSY_H */
