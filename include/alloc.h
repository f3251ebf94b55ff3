/*
 * alloc.h - C ABI of the layer allocator (host code, no device work).
 *
 * Paper section IV: before training, a central server places the L layers
 * of the model on D devices as contiguous blocks, device i holding layers
 * pi[i] .. pi[i+1]-1 (the partition index, an array of D+1 integers with
 * pi[0] = 0 and pi[D] = L).  Its inputs come from two benchmarks
 * (section IV-B): per device the time ratio dt, the available memory dm and
 * the communication time ct; per layer the FLOPs lf and the memory lm.
 * The allocation is a mixed-integer program (section IV-C); section IV-D
 * replaces it with a two-stage heuristic, implemented here:
 *   alloc_coarse  - Algorithm 1, coarse allocation by memory;
 *   alloc_fine    - Algorithm 2, workload fine-tuning;
 *   alloc_workloads evaluates a partition.
 *
 * Conventions
 *   - All arrays are host memory owned by the caller; the library keeps no
 *     state between calls and allocates nothing the caller must free.
 *   - Units are the caller's: lm and dm in one memory unit, dt * lf and ct
 *     in one time unit.  All values must be finite; dt, lf, lm >= 0,
 *     ct >= 0, dm >= 0.
 *   - Every call returns an alloc_status and never aborts or throws.
 *   - Workload of device i (section IV-D): each of its layers j costs
 *     dt[i] * lf[j] + ct[i], and the device's workload is the sum over its
 *     layers.  (The program of section IV-C charges ct[i] once per device;
 *     alloc_workloads reports either form.)
 */
#ifndef SKY_ALLOC_H
#define SKY_ALLOC_H

#ifdef __cplusplus
extern "C" {
#endif

/* Enumerations are int-sized on both sides of the ABI.  Compiled as C++
 * they get a fixed underlying type int, so that every int a C caller passes
 * is a value of the type there too (and is rejected by the argument checks
 * when it is not one of the listed values), instead of being undefined. */
#ifndef SKY_ENUM_INT
#ifdef __cplusplus
#define SKY_ENUM_INT : int
#else
#define SKY_ENUM_INT
#endif
#endif

typedef enum SKY_ENUM_INT {
  ALLOC_OK = 0,
  ALLOC_EINVAL = 1, /* L < D, D < 1, null pointer, non-finite or negative input,
                       malformed partition index */
  ALLOC_ENOFIT = 2  /* Algorithm 1 cannot meet every device's memory: a full
                       sweep left the partition index unchanged (or it kept
                       changing for L * D sweeps) */
} alloc_status;

typedef enum SKY_ENUM_INT {
  ALLOC_CT_PER_LAYER = 0, /* sum_j (dt[i] lf[j] + ct[i]), section IV-D */
  ALLOC_CT_PER_DEVICE = 1 /* dt[i] sum_j lf[j] + ct[i], section IV-C */
} alloc_ct_mode;

/*
 * Algorithm 1 (section IV-D, coarse allocation by memory).  Starts from the
 * equal split pi[i] = floor(i L / D) and sweeps devices 0 .. D-2: while
 * device i holds more memory than dm[i] and more than one layer it hands its
 * last layer to device i+1; then, while the next layer would still fit in
 * dm[i] (strictly) and device i+1 keeps more than one layer, it takes device
 * i+1's first layer.  Stops when every device's layers fit (ALLOC_OK) or a
 * sweep changes nothing (ALLOC_ENOFIT).
 *   lm: [L] layer memory; dm: [D] device memory;
 *   pi_out: [D+1] partition index (written on ALLOC_OK and ALLOC_ENOFIT:
 *   the last state); sweeps: if not NULL, the number of sweeps run.
 */
alloc_status alloc_coarse(int L, int D, const double* lm, const double* dm, int* pi_out,
                          int* sweeps);

/*
 * Algorithm 2 (section IV-D, workload fine-tuning) on a partition that meets
 * the memory limits (e.g. alloc_coarse's).  Each round sets the target to
 * the mean device workload (ALLOC_CT_PER_LAYER form) and sweeps i = 0 .. D-2
 * on the current partition: if device i is below the target, device i+1
 * keeps more than one layer and device i's memory allows it, device i takes
 * device i+1's first layer; otherwise, if device i+1 is below the target,
 * device i minus its last layer's workload is still above the target, device
 * i keeps more than one layer and device i+1's memory allows it, device i
 * hands its last layer to device i+1.  Returns after a round that changes
 * nothing or after max_iter rounds.
 *   pi: [D+1] in: starting partition, out: tuned partition;
 *   rounds: if not NULL, the number of rounds run.
 */
alloc_status alloc_fine(int L, int D, const double* dt, const double* dm, const double* ct,
                        const double* lf, const double* lm, int max_iter, int* pi, int* rounds);

/*
 * Workload of every device under partition pi: w_out[i] for i < D.
 * EINVAL for a mode other than the two alloc_ct_mode values.
 * Rejects a pi that is not 0 = pi[0] < pi[1] < ... < pi[D] = L.
 */
alloc_status alloc_workloads(int L, int D, const double* dt, const double* ct, const double* lf,
                             const int* pi, alloc_ct_mode mode, double* w_out);

#ifdef __cplusplus
}
#endif

#endif /* SKY_ALLOC_H */
