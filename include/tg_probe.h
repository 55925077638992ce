/*
 * libtg_probe.so: measurement helper of the benchmark, not part of the stitching path.
 *
 * A plain streaming kernel that reads `read_bytes` and writes `write_bytes` with 16-byte
 * nontemporal stores, so that the stitch kernel's HBM rate can be set beside what the
 * memory system delivers to a kernel with no work of its own for the same mix of reads
 * and writes. Each workgroup reads one chunk and writes one chunk of `chunk` bytes (the
 * read chunk scaled by read_bytes / write_bytes); workgroups take chunks in address order.
 */
#ifndef TG_PROBE_H
#define TG_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* src: device, >= read_bytes; dst: device, >= write_bytes; both 16-byte aligned, sizes
 * multiples of 16, chunk a multiple of 4096. Enqueued on `stream`. Returns 0, or -1 for
 * bad arguments, -2 when the launch fails. */
int tg_probe_stream(const void *src, int64_t read_bytes, void *dst, int64_t write_bytes,
                    int32_t chunk, void *stream);

/* The same with the written bytes cut into `planes` equal planes (1..4; write_bytes a
 * multiple of 16 * planes) and each workgroup writing its chunk as `planes` equal runs at
 * the same offset in every plane, as a stitch work unit writes the three fp16 planes of
 * its rows. planes == 1 is tg_probe_stream. Same arguments and returns otherwise. */
int tg_probe_stream_planes(const void *src, int64_t read_bytes, void *dst, int64_t write_bytes,
                           int32_t chunk, int32_t planes, void *stream);

/* Replay of one stitch launch's memory traffic with no work of its own: workgroup g
 * (of n_units, units_per_canvas per canvas) reads the 16-byte words of src covering the
 * byte ranges [off[k], off[k] + len[k]) for k in [begin[g], begin[g+1]) (the source rows
 * of the patches in stitch unit g, as tg_stitch reads them), then writes unit g's
 * run_bytes (the last unit of a canvas: the rest of the plane) of each of its canvas's
 * three planes of plane_bytes, canvases of three planes from dst, with 16-byte nontemporal
 * stores. off, len, begin: device; every range must lie in src's first src_bytes, rounded
 * up to 16 (the caller checks). Returns 0, -1 for bad arguments, -2 when the launch
 * fails. */
int tg_probe_replay(const void *src, int64_t src_bytes, const int64_t *off, const int32_t *len,
                    const int32_t *begin, int32_t n_units, int32_t units_per_canvas, void *dst,
                    int64_t plane_bytes, int64_t run_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* TG_PROBE_H */
