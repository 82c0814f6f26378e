/*
 * esp_calib.h -- measurement kernel of the Elastic Shadow Pricing library
 * (libesp_calib.so, built beside libesp.so).  Not part of the method and not
 * used by it: it times the memory system on the access pattern of the fused
 * price-iteration kernel, to give that kernel's roofline an achievable
 * ceiling measured on the same machine.
 */
#ifndef ESP_CALIB_H
#define ESP_CALIB_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * esp_calib_stream: enqueue one read-only pass over a table laid out like one
 * cluster of the packed table (ncol fp32 columns, column c starting at
 * table + c * col_len, tiles of 256 entries), on `blocks` workgroups of 4
 * wavefronts, with the fused dense kernel's load pattern (one 128-bit
 * non-temporal load per lane per column per tile, three tiles in registers,
 * loads past the end clamped to the last tile).
 *   table   device, ncol * col_len floats (any values)
 *   ncol    1..10;  col_len >= tiles * 256;  tiles >= 1;  blocks >= 1
 *   sink    device, blocks * 256 floats: one value per thread (keeps the loads
 *           alive; its contents are meaningless)
 *   stream  hipStream_t (NULL = the null stream)
 * Returns 0, 1 for bad arguments (nothing enqueued), 8 when the launch failed.
 */
int esp_calib_stream(const float *table, int ncol, size_t col_len, int tiles, int blocks, float *sink, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* ESP_CALIB_H */
