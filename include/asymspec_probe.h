/*
 * asymspec_probe.h -- read-ceiling and core-clock probes for MI355X (gfx950),
 * built as libasymspec_probe.so beside libasymspec.so.
 *
 * Not part of the decision step.  It measures how fast a plain kernel can
 * stream a buffer from HBM with the same 16-byte non-temporal loads the
 * decision kernel uses, so that the decision kernel's achieved bandwidth can
 * be reported both as a fraction of the 8 TB/s specification and as a
 * fraction of this measured ceiling (the decision step itself is bound by HBM
 * reads: every logit is read once, and nothing forms a dense contraction).
 */
#ifndef ASYMSPEC_PROBE_H_
#define ASYMSPEC_PROBE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ASYMSPEC_PROBE_E_ARG (-1)       /* invalid argument; nothing enqueued */
#define ASYMSPEC_PROBE_E_DEVICE (-2)    /* the launch failed */
#define ASYMSPEC_PROBE_MAX_BLOCKS (1 << 20)
#define ASYMSPEC_PROBE_MAX_CLOCK_BLOCKS 4096
#define ASYMSPEC_PROBE_MAX_CLOCK_TICKS 1000000u   /* 10 ms of the 100 MHz counter */

/*
 * Reads nbytes of device memory at src once and writes, for each of the
 * nblocks workgroups, the XOR of every 32-bit word that workgroup read into
 * out[workgroup].  The XOR of all of out[0..nblocks) equals the XOR of every
 * 32-bit word of the buffer (the check that the whole buffer was read).
 *
 *   src      device pointer, 16-byte aligned, owned by the caller, not written
 *   nbytes   a multiple of 16, in [16, 2^40]
 *   out      device pointer to nblocks uint32 words, 4-byte aligned, overwritten
 *   nblocks  workgroups of 256 threads in [1, ASYMSPEC_PROBE_MAX_BLOCKS];
 *            they stride over the buffer, 32 KiB per workgroup per step
 *   stream   hipStream_t to enqueue on (NULL: the default stream)
 *
 * Asynchronous: returns once the kernel is enqueued.  Returns 0, or
 * ASYMSPEC_PROBE_E_ARG (checked on the host before any device work) or
 * ASYMSPEC_PROBE_E_DEVICE.  The library allocates nothing.
 */
int asymspec_probe_read(const void* src, size_t nbytes, uint32_t* out, int nblocks, void* stream);

/*
 * Samples the core (shader) clock: each of nblocks single-wave workgroups
 * waits `ticks` ticks of the GPU's constant 100 MHz real-time counter and
 * writes the shader-clock cycles that elapsed meanwhile to out[2 k] and the
 * real-time ticks to out[2 k + 1] (k the workgroup).  The clock of workgroup
 * k in MHz is 100 * out[2 k] / out[2 k + 1].  Used to record the clock
 * around timed regions (the decision step's ALU work scales with it).
 *
 *   out      device pointer to 2 * nblocks uint32 words, 4-byte aligned, overwritten
 *   nblocks  in [1, ASYMSPEC_PROBE_MAX_CLOCK_BLOCKS]
 *   ticks    in [1, ASYMSPEC_PROBE_MAX_CLOCK_TICKS]
 *   stream   hipStream_t to enqueue on (NULL: the default stream)
 *
 * Asynchronous; returns 0, ASYMSPEC_PROBE_E_ARG (checked on the host, nothing
 * enqueued) or ASYMSPEC_PROBE_E_DEVICE.
 */
int asymspec_probe_clock(uint32_t* out, int nblocks, uint32_t ticks, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ASYMSPEC_PROBE_H_ */
