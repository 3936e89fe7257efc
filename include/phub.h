/*
 * phub.h - C interface of the PHub gradient-exchange step on one MI355X GPU.
 *
 * The paper (Parameter Hub, section 3.1) states the service as: create a
 * job handle and namespace, initialise receive and merge buffers, then let
 * workers Push gradients for keys and Pull the updated model.  Between push
 * and pull the server aggregates every key's gradients over all workers and
 * runs the optimizer on the result (section 3.2.2), chunk by chunk (section
 * 3.2.3), with chunks mapped to cores by a schedule fixed at initialisation
 * (section 3.2.4).
 *
 * Here the server is one GPU.  The N workers' gradients are device buffers
 * that the caller owns; a push registers a pointer and copies nothing.  One
 * step runs one fused kernel over all keys: it sums the N gradients of each
 * element in ascending worker order in fp32 and applies momentum or
 * Nesterov SGD with coupled weight decay to the job's master weights and
 * momentum, reading each gradient byte once.
 *
 * Per element, with s the sum, w the weight and m the momentum, each line a
 * single fused multiply-add rounded once to fp32:
 *     d  = wd * w + s
 *     m' = mu * m + d
 *     u  = mu * m' + d     (Nesterov)   or   u = m'   (plain momentum)
 *     w' = -lr * u + w
 *
 * Conventions for every function below:
 *   - the return value is PHUB_OK (0) or a negative PHUB_E* code; no
 *     exception or signal crosses this interface;
 *   - on an error nothing is enqueued or changed, and phub_last_error()
 *     returns a message for the calling thread;
 *   - "device pointer" means memory of the GPU that was current when the job
 *     was created (torch tensors' data_ptr(), hipMalloc memory);
 *   - calls on one job must not overlap; different jobs may be driven from
 *     different threads.
 */
#ifndef PHUB_H
#define PHUB_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum phub_status {
    PHUB_OK = 0,
    PHUB_EINVAL = -1,    /* an argument is out of range, null or misaligned */
    PHUB_ENOTREADY = -2, /* phub_step before every (worker, key) was pushed */
    PHUB_ENOMEM = -3,    /* device or host allocation failed */
    PHUB_EHIP = -4,      /* a HIP runtime call failed (message names it) */
    PHUB_ESTATE = -5     /* the handle is not a live job */
};

/* One training job: a namespace of keys, its workers, master weights and
 * momentum (the handle of section 3.1).  Opaque. */
typedef struct phub_job phub_job;

/*
 * phub_init - create a job (section 3.1: CreateService + InitService).
 *   out           receives the new handle.
 *   num_workers   N, 1 <= N <= 4096: the number of gradients summed per key.
 *   num_keys      K >= 1: the number of keys (one layer's parameters each,
 *                 section 2).
 *   key_elems     host array of K element counts, each 0 <= n_k < 2^34
 *                 (the schedule functions below accept up to 2^40).
 *   chunk_bytes   size of the chunks keys are split into for scheduling
 *                 (section 3.2.3; the paper's default is 32768); a positive
 *                 multiple of 16, at most 2^30.  Results do not depend on it.
 *   lr, momentum, weight_decay
 *                 optimizer settings (section 4.2), finite fp32 values, kept
 *                 for the life of the job.
 *   nesterov      nonzero for Nesterov momentum, zero for plain momentum.
 *   hip_stream    the hipStream_t all of the job's device work is ordered
 *                 on, or NULL to let the job create its own non-blocking
 *                 stream (destroyed with the job).  A caller's stream is
 *                 borrowed and must outlive the job.
 * The job allocates its master weights W and momentum M (fp32, each key's
 * slice 256-byte aligned), sets both to zero, computes the chunk schedule
 * (section 3.2.4) and uploads it.  Errors: PHUB_EINVAL, PHUB_ENOMEM,
 * PHUB_EHIP.  On error *out is set to NULL.
 */
int phub_init(phub_job **out, int num_workers, int num_keys, const int64_t *key_elems,
              int64_t chunk_bytes, float lr, float momentum, float weight_decay,
              int nesterov, void *hip_stream);

/* Chunk-to-wave schedules (section 3.2.4; see the schedule section below). */
enum phub_schedule {
    PHUB_SCHEDULE_SPLIT = 0,  /* contiguous, exactly balanced runs of chunks */
    PHUB_SCHEDULE_LPT = 1,    /* the paper's balanced partition of chunks (default) */
    PHUB_SCHEDULE_DYNAMIC = 2 /* phub_init_ex only: the LPT schedule, except that the
                                 streamed state's full 1024-element tiles are not fixed
                                 per wave: each launch's waves take them one at a time,
                                 in address order, from a counter they share (work
                                 stealing), so that waves that start late take fewer.
                                 Kept for jobs with a fixed-N kernel (1-16, 20, 24 or
                                 32 workers, fused); others run as LPT. */
};

/* Optimizers (section 3.2.2: aggregators and optimizers are pluggable).
 * All take the same aggregated gradient s and coupled L2 weight decay wd:
 * d = s + wd*w. */
enum phub_optimizer {
    PHUB_OPT_MOMENTUM = 0, /* SGD with momentum: phub_init's momentum and
                              nesterov arguments (section 4.2; default) */
    PHUB_OPT_SGD = 1,      /* plain SGD, no state: w' = w - lr*d */
    PHUB_OPT_ADAM = 2      /* Adam with bias correction (beta1, beta2, eps
                              below; state M and V); the step number t counts
                              the job's completed phub_step calls, from 1 */
};

/* Optional settings of phub_init_ex. */
typedef struct phub_options {
    int schedule;           /* a phub_schedule value */
    int64_t resident_bytes; /* cache budget in bytes for this job's optimizer
                               state (the paper's cached model, section 4.5).
                               The state of the arena's first
                               floor(budget / (4 S)) elements (S state arrays,
                               4 bytes each), cut back to a tile boundary
                               (1024 elements) inside the key that crosses
                               that point, is read and written with the
                               cache-allocating policy so that it can stay in
                               the GPU's memory-side cache between steps; the
                               rest streams non-temporally like the
                               gradients.  0: nothing is cached; a budget at
                               least the state's size caches all of it.  -1:
                               the default, a per-device budget of 256 MiB
                               (the memory-side cache of MI355X) shared first
                               come, first served by the live jobs created
                               with -1 (each takes what its state needs of
                               what is left) and given back by phub_destroy;
                               jobs whose streamed state is written back in
                               bursts take none of it (they stream as fast as
                               they cache): momentum SGD and plain SGD with
                               6 to 16, 20, 24 or 32 workers, Adam with 14 to
                               16, 20, 24 or 32, not unfused.  A job that
                               will step with pushpull (whose kernels write
                               the model buffers and have no burst
                               write-back) gains from an explicit budget:
                               measured 0.81 against 0.70 of peak for 8
                               workers over 25.6 M parameters with all of its
                               state cached.  Results do not depend on it. */
    int num_groups;         /* readiness groups (sections 3.2.2-3.2.3: a
                               chunk is aggregated as soon as all of its
                               pieces have arrived).  0: none; the whole step
                               is enqueued by phub_step.  > 0: key k belongs
                               to group key_group[k]; as soon as every worker
                               has pushed every key of a group, that group's
                               aggregation and update are enqueued on the
                               job's stream (after a device-side wait on the
                               ready events of its pushes), while later
                               groups are still being pushed.  Results do not
                               depend on the grouping. */
    const int *key_group;   /* num_keys entries in [0, num_groups), read
                               during phub_init_ex only; ignored when
                               num_groups is 0. */
    int optimizer;          /* a phub_optimizer value (0: momentum SGD) */
    float beta1, beta2;     /* Adam: moment decay rates, each in [0, 1) */
    float eps;              /* Adam: added to the root of the second moment
                               (finite, >= 0).  The three are ignored by the
                               other optimizers; momentum and nesterov of
                               phub_init_ex are ignored by SGD and Adam. */
    int workgroups;         /* persistent workgroups of the job's launch (each
                               a wave per SIMD of one compute unit), at most
                               65536; 0: one per compute unit.  Fewer let concurrent
                               tenants share the chip without each keeping a
                               full grid of loads in flight. */
    int unfused;            /* ablation of the fused pass (section 3.2.2:
                               the aggregating thread also optimizes): 1
                               runs the step as two launches, a sum of the N
                               gradients into a job-owned merge buffer, then
                               the optimizer over it ((N + 6) * 4 bytes per
                               element instead of (N + 4) * 4).  Same
                               results.  Not with readiness groups or
                               pushpull (PHUB_EINVAL).  0: fused (default). */
    int ordered_events;     /* 1: the caller guarantees that each worker's
                               ready events (phub_push_event and the batched
                               forms) are recorded on one stream, in the
                               order of its pushes; a launch then waits only
                               for each worker's last event among the keys it
                               covers (at most num_workers waits instead of
                               one per distinct event; each wait costs device
                               time when it resolves).  0 (default): every
                               distinct event is waited for.  Either way,
                               events already complete when the launch is
                               enqueued are not waited for. */
    int whole_chunks;       /* ablation of the chunk size (section 3.2.3):
                               1 keeps every chunk of chunk_bytes an
                               indivisible item of the LPT schedule, as in
                               the paper (no splitting of chunks however few
                               they are).  0 (default): while there are fewer
                               than 128 items per wave, chunks are halved, not
                               below 1024 elements, so that every wave has
                               work.  Results do not depend on it. */
} phub_options;

/*
 * phub_init_ex - phub_init with options (NULL means the defaults: LPT
 * schedule, shared cache budget).  Errors as phub_init, plus PHUB_EINVAL for
 * an unknown schedule or resident_bytes < -1.
 */
int phub_init_ex(phub_job **out, int num_workers, int num_keys, const int64_t *key_elems,
                 int64_t chunk_bytes, float lr, float momentum, float weight_decay,
                 int nesterov, void *hip_stream, const phub_options *options);

/*
 * phub_set_weights - load key `key`'s master weights from `src` (n_k fp32
 * values, device or host memory) and reset its momentum to zero.  The copy
 * is ordered on the job's stream; `src` must stay valid until it has run
 * (phub_sync).  Errors: PHUB_EINVAL, PHUB_ESTATE, PHUB_EHIP.
 */
int phub_set_weights(phub_job *job, int key, const float *src);

/*
 * phub_push - worker `worker` pushes its gradient for key `key` (section
 * 3.1 Push; zero-copy registration as in section 3.2.1).
 *   grad   device pointer to n_k fp32 values, 16-byte aligned (may be NULL
 *          only when n_k == 0).  The caller keeps ownership; the buffer must
 *          stay valid and unchanged until the step that consumes it has run
 *          on the job's stream.
 * Nothing is copied: the pointer is recorded for the next phub_step.  The
 * worker index, not the call order, fixes the worker's place in the sum.
 * Pushing a pair again before the step replaces the earlier pointer.  With
 * readiness groups, the push that completes a group enqueues that group's
 * work (see phub_options.num_groups); pushing a key of a group that has
 * already been enqueued in this step is PHUB_ESTATE.
 * Errors: PHUB_EINVAL (range, null, alignment), PHUB_ESTATE, PHUB_EHIP (an
 * enqueue triggered by the push failed).
 */
int phub_push(phub_job *job, int worker, int key, const float *grad);

/*
 * phub_push_event - phub_push for a gradient that is still being produced:
 * it is ready once `hip_event` (a hipEvent_t recorded by the producer on its
 * own stream; NULL = ready now) has completed.  The step's work that reads
 * this gradient waits for the event on the device (hipStreamWaitEvent on the
 * job's stream); the host never blocks on it.  The event must stay valid
 * until that work is enqueued: when its readiness group completes, at the
 * latest at phub_step.  Same rules and errors as phub_push.
 */
int phub_push_event(phub_job *job, int worker, int key, const float *grad, void *hip_event);

/*
 * phub_push_keys - batched phub_push for one worker: pushes grads[i] for key
 * keys[i], i < count (keys == NULL means keys 0 .. count-1).  Same rules as
 * phub_push; either every pointer is recorded or, on an argument error,
 * none is.
 */
int phub_push_keys(phub_job *job, int worker, int count, const int *keys,
                   const float *const *grads);

/*
 * phub_push_all - every worker pushes every key in one call (section 3.1's
 * Push, for a caller that holds all of a step's gradients): grads has
 * num_workers * num_keys entries, grads[w * num_keys + k] being worker w's
 * gradient for key k (host array of device pointers, read during the call
 * only).  Same rules and errors as phub_push for each entry; either every
 * pointer is recorded or, on an argument error (PHUB_EINVAL) or when a
 * readiness group has already been enqueued this step (PHUB_ESTATE), none
 * is.  With readiness groups, every group is enqueued during the call.
 */
int phub_push_all(phub_job *job, const float *const *grads);

/*
 * phub_push_keys_event - phub_push_keys whose gradients are all ready once
 * `hip_event` has completed (as phub_push_event; NULL = ready now): one call
 * per worker for a bucket of keys that one producer event covers.  Either
 * every pointer is recorded or, on an argument error, none is; a group
 * completed part-way through the call is enqueued at that point.
 */
int phub_push_keys_event(phub_job *job, int worker, int count, const int *keys,
                         const float *const *grads, void *hip_event);

/*
 * phub_pushpull - PushPull (section 3.1): push worker `worker`'s gradient
 * for key `key` (as phub_push) and have the step write the key's updated
 * weights into `model_out` (n_k fp32 values, 16-byte aligned, caller-owned;
 * must not overlap any gradient, W, M or another model buffer).  The copy is
 * written by the same fused pass that updates W, right after each piece of
 * the key is optimized, so W is not read again to broadcast it.  The buffer
 * is filled once the step has run on the job's stream (phub_sync, or an
 * event recorded on the job's stream after phub_step).  The registration
 * lasts for this step only.  In a step, or in a readiness group, either
 * every (worker, key) pair gives a model buffer or none does: a mix is
 * PHUB_EINVAL when the step (or the group) is enqueued, and nothing of it is
 * enqueued.  Errors: as phub_push, and PHUB_EINVAL for a null or misaligned
 * model_out.
 */
int phub_pushpull(phub_job *job, int worker, int key, const float *grad, float *model_out);

/*
 * phub_pushpull_keys - batched phub_pushpull for one worker, all gradients
 * ready once `hip_event` has completed (NULL = ready now): grads[i] and
 * model_outs[i] for key keys[i], i < count (keys == NULL means keys
 * 0 .. count-1).  Argument errors are found before anything is recorded.
 */
int phub_pushpull_keys(phub_job *job, int worker, int count, const int *keys,
                       const float *const *grads, float *const *model_outs, void *hip_event);

/*
 * phub_step - aggregate and optimize every key (sections 3.2.2-3.2.4): one
 * kernel launch over all keys on the job's stream, asynchronous to the
 * host.  Requires every (worker, key) pair to have been pushed since the
 * previous step, else PHUB_ENOTREADY and nothing is enqueued.  If a pushed
 * pointer differs from the last step's, the pointer table is uploaded on the
 * same stream first; the launch first waits for the ready events given to
 * phub_push_event.  Afterwards all pairs count as not pushed.
 * With readiness groups, the groups were enqueued as they completed; the
 * step enqueues any group without keys, closes the step, and reports
 * PHUB_ENOTREADY (enqueuing nothing more) while a pair is missing: the groups
 * already enqueued stay applied, and the step completes once the missing
 * pushes arrive and phub_step is called again.
 * With pushpull registrations (phub_pushpull), the same pass also writes
 * each key's updated weights into every worker's model buffer.
 * Errors: PHUB_ENOTREADY, PHUB_EINVAL (a mix of pushes with and without a
 * model buffer), PHUB_ESTATE, PHUB_EHIP.
 */
int phub_step(phub_job *job);

/*
 * phub_pull - the current master weights of key `key` (section 3.1 Pull):
 * *weights receives a device pointer to n_k fp32 values owned by the job.
 * Reads are ordered after earlier steps on the job's stream (phub_sync
 * before reading from another stream or the host); the values change at the
 * next phub_step and the pointer is valid until phub_destroy.
 * Errors: PHUB_EINVAL, PHUB_ESTATE.
 */
int phub_pull(phub_job *job, int key, const float **weights);

/*
 * phub_get_state - device pointers to key `key`'s master weights and
 * momentum (Adam: first moment; plain SGD: NULL), n_k fp32 each,
 * job-owned, same validity as phub_pull.  Either output may be NULL.
 * Errors: PHUB_EINVAL, PHUB_ESTATE.
 */
int phub_get_state(phub_job *job, int key, const float **weights, const float **momentum);

/*
 * phub_get_second_moment - device pointer to key `key`'s second moment
 * (Adam), or NULL for the other optimizers.  Errors: PHUB_EINVAL,
 * PHUB_ESTATE.
 */
int phub_get_second_moment(phub_job *job, int key, const float **second);

/*
 * phub_sync - wait on the host until all work enqueued by the job has run.
 * Errors: PHUB_ESTATE, PHUB_EHIP (including faults of earlier launches).
 */
int phub_sync(phub_job *job);

/*
 * phub_get_stream - the hipStream_t the job orders its work on.
 */
int phub_get_stream(phub_job *job, void **hip_stream);

/*
 * phub_job_info - launch shape of the job's step: the number of workgroups
 * of one launch (0 if every key is empty), the threads per workgroup, the
 * number of work segments in the schedule, the bytes of optimizer state
 * (S arrays over the padded arena), and how many of those bytes are
 * scheduled as cache-resident (0: all of the state streams non-temporally;
 * equal to the state bytes, less the padding, when all of it is cached).
 * Any output may be NULL.
 */
int phub_job_info(phub_job *job, int *workgroups, int *threads_per_group, int64_t *segments,
                  int64_t *state_bytes, int64_t *resident_bytes);

/*
 * phub_destroy - wait for the job's work, free its memory (W, M, schedule,
 * pointer table) and its own stream.  The handle is dead afterwards; passing
 * it again to any function returns PHUB_ESTATE.
 */
int phub_destroy(phub_job *job);

/*
 * phub_step_noalloc - one exchange step that allocates no memory: for
 * callers that cannot allocate device memory (serving loops that must not
 * call hipMalloc, harnesses that forbid allocation).  It computes what
 * phub_init + phub_push_all + phub_step compute for one step of a momentum
 * job created with the same arguments, on caller-owned state.
 *   num_workers, num_keys, key_elems, chunk_bytes, lr, momentum,
 *   weight_decay, nesterov
 *                 as phub_init (same limits).
 *   grads         host array of num_workers * num_keys device pointers,
 *                 grads[w * num_keys + k] worker w's gradient for key k (as
 *                 phub_push_all); read during the call only.
 *   weights, moments
 *                 device arenas of W and M (fp32, 16-byte aligned), updated
 *                 in place, laid out like a job's state: key k starts at
 *                 element A_k = sum over j < k of n_j rounded up to a
 *                 multiple of 64; the padding is neither read nor written.
 *                 NULL only when every key is empty.
 *   hip_stream    the hipStream_t the step is ordered on (NULL = the null
 *                 stream).
 * The step's schedule and pointer table live in a device array of the
 * library of 4 MiB (PHUB_NOALLOC_SCRATCH_BYTES), one per GPU, held until
 * the process ends; that bounds a call to about 240 M parameters and
 * PHUB_EINVAL reports a step that does not fit, before anything is
 * enqueued.  The call uploads the schedule on hip_stream after the stream's
 * earlier work and waits for that upload (the host thread blocks until the
 * stream's earlier work is done); the kernel itself runs asynchronously.
 * Calls on one GPU share its array: calls that overlap on one GPU (from
 * other threads, or on another stream before this call's kernel has run)
 * race and give wrong results.  All state streams non-temporally (nothing
 * is kept in the memory-side cache).  Errors: PHUB_EINVAL, PHUB_ENOMEM (host
 * memory), PHUB_EHIP.
 */
int phub_step_noalloc(int num_workers, int num_keys, const int64_t *key_elems,
                      int64_t chunk_bytes, float lr, float momentum, float weight_decay,
                      int nesterov, const float *const *grads, float *weights, float *moments,
                      void *hip_stream);

/* Message of the last failed call on this thread ("" if none).  The string
 * belongs to the library and lives until the thread's next failing call. */
const char *phub_last_error(void);

/* --------------------------------------------------------------------------
 * The chunk schedule (section 3.2.4), computed on the host only.  phub_init
 * runs it; it is exported so that its coverage and balance can be checked
 * without a GPU.
 *
 * The unit that plays a PHub core is one wave (64 lanes) of the fused
 * kernel; the kernel runs one persistent workgroup per compute unit, and
 * each wave walks its own bin: a list of segments fixed at initialisation.
 * Keys are cut into chunks of chunk_bytes/4 elements (section 3.2.3's
 * virtual keys), the last one of a key partial.
 *
 * PHUB_SCHEDULE_SPLIT: the keys, in key order, are dealt to the num_bins
 *   bins as contiguous runs of equal length (to within one 16-byte float4),
 *   each run cut into segments at chunk boundaries.  On a GPU a chunk can be
 *   split on any 16-byte boundary, so the load is balanced exactly.  All
 *   num_bins bins are kept (an empty run is an empty bin); min_items is
 *   ignored.
 * PHUB_SCHEDULE_LPT: chunks are indivisible items, as in the paper.  Keys
 *   smaller than a chunk are bundled, in key order, into items of at most one
 *   chunk (a run of small keys is not bundled across a larger key).  While
 *   there are fewer than min_items items, the chunk is halved (not below
 *   1024 elements).  Items go to the bins by the longest-processing-time-
 *   first rule (largest item first, each to the least loaded bin, lowest
 *   index on ties), a 4/3-approximate balanced partition like the paper's.
 *   Bins that get no item are dropped.
 * Item and segment cost is the bytes moved, (N + 4) * 4 per element, plus
 * 4096 per segment.  The result of a step depends on neither schedule nor
 * chunk size.  phub_init uses one bin per wave of its launch (one workgroup
 * of 4 waves per compute unit) and, for LPT, min_items = 32 per bin.
 * ------------------------------------------------------------------------ */

/* One contiguous run of one key handled by one wave. */
typedef struct phub_segment {
    int32_t key;    /* key index */
    int32_t count;  /* number of elements, >= 1 */
    int64_t offset; /* index of the first element within the key, a multiple of 4 */
} phub_segment;

/*
 * phub_plan_count - sizes of the schedule for these arguments (same meaning
 * and checks as phub_init; schedule a phub_schedule value; num_bins >= 1;
 * min_items >= 0): *num_segments, *bins_used and *item_elems (the chunk
 * size after refinement).  Any output may be NULL.  Errors: PHUB_EINVAL.
 */
int phub_plan_count(int num_workers, int num_keys, const int64_t *key_elems,
                    int64_t chunk_bytes, int schedule, int num_bins, int min_items,
                    int64_t *num_segments, int *bins_used, int64_t *item_elems);

/*
 * phub_plan_build - the schedule itself, into caller arrays sized by
 * phub_plan_count: segments[num_segments], grouped by bin;
 * bin_begin[bins_used + 1], bin b owning segments bin_begin[b] ..
 * bin_begin[b+1]-1 in key, then offset, order; bin_cost[bins_used] (may be
 * NULL) the cost of each bin.  Errors: PHUB_EINVAL.
 */
int phub_plan_build(int num_workers, int num_keys, const int64_t *key_elems,
                    int64_t chunk_bytes, int schedule, int num_bins, int min_items,
                    phub_segment *segments, int64_t *bin_begin, int64_t *bin_cost);

#ifdef __cplusplus
}
#endif

#endif /* PHUB_H */
