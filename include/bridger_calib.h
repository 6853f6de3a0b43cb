/*
 * bridger_calib.h -- calibration microbenchmarks (libbridger_calib.so).
 *
 * The data-movement model of Eq. 1 (Sec. 4.5) takes, for every memory level l, a bandwidth
 * BandWidth_l and a capacity Capacity_l of the target device (Table 6).  These calls measure
 * the bandwidths that bound batched tree-ensemble prediction on the current device: the rate
 * of per-lane LDS gathers (every internal-node visit of the traversal kernels takes two of
 * them, the node record and the row's feature value), the rate of per-lane gathers from the
 * L2 (the node records of forests too large for the LDS), and the HBM copy rate.  They are not
 * part of prediction and the prediction library does not call them; the benchmark uses them
 * to show that the peak it rates the kernels against holds on the device.
 *
 * Every call runs on the current device and the null stream, allocates and frees its own
 * device buffers, synchronizes, and returns 0 or a hipError_t code.  Output pointers may be
 * NULL.
 */
#ifndef BRIDGER_CALIB_H
#define BRIDGER_CALIB_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Compute units, the peak engine clock (kHz) and the LDS bytes per compute unit, as the
 * runtime reports them. */
int bridger_calib_device(int32_t *n_cu, int32_t *max_clock_khz, int32_t *lds_bytes_per_cu);

/*
 * Per-lane LDS gathers of width_bytes (4, 8 or 16) per lane: 32 resident waves per compute
 * unit, every lane issuing 16 independent reads per iteration at addresses held in a
 * register.  distinct = 64 gives every lane its own element, the 32 lanes of each half-wave on
 * distinct banks (a permuted lane order, as the traversal kernels' feature tile does);
 * distinct = 1, 2, 4, ..., 32 lets the lanes share that many elements (as a wave's lanes share
 * the node records of a tree's upper levels); distinct = 0 draws the addresses at random from
 * a 1 KB window (bank conflicts).  Other values: hipErrorInvalidValue.  Timed over `reps`
 * launches after ten untimed ones.  *wave_reads_per_s counts wave-wide read instructions per
 * second over the whole device; divide by the compute units and the clock for instructions
 * per clock per CU, and multiply by 64 for lanes.
 */
int bridger_calib_lds_gather(int32_t width_bytes, int32_t distinct, int32_t reps,
                             double *ms_per_launch, double *wave_reads_per_s);

/*
 * Per-lane global-memory gathers of width_bytes (4, 8 or 16) per lane from a device buffer of
 * 2^buffer_log2 bytes (16..30; 2 MiB and below stay in the L2): 32 resident waves per compute
 * unit, every lane issuing 16 independent loads per iteration, each iteration on new cache
 * lines of the buffer (the global-node traversal kernels read their node records this way).
 * distinct = 64 puts every lane of a wave on its own 128-byte line; distinct = 1, 2, ..., 32
 * lets the lanes share that many lines.  Other values: hipErrorInvalidValue.  Timed over
 * `reps` launches after ten untimed ones; *wave_loads_per_s counts wave-wide load
 * instructions per second over the whole device.
 */
int bridger_calib_global_gather(int32_t width_bytes, int32_t distinct, int32_t buffer_log2,
                                int32_t reps, double *ms_per_launch, double *wave_loads_per_s);

/* A plain 16-byte-per-lane device-to-device copy of `bytes` bytes (two buffers of that size),
 * timed over `reps` launches after ten untimed ones; *bytes_per_s counts bytes read plus
 * bytes written. */
int bridger_calib_copy(int64_t bytes, int32_t reps, double *ms_per_copy, double *bytes_per_s);

#ifdef __cplusplus
}
#endif

#endif /* BRIDGER_CALIB_H */
