/*
 * schedprobe.h -- throughput probes for the roofline of the simulator
 * (libschedprobe.so; measurement infrastructure, not part of the simulator).
 *
 * The simulation kernel is priced against the chip's 32-bit integer VALU
 * peak (256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz = 39.3e12 lane-operations/s)
 * and its LDS bandwidth (128 B per clock per CU = 78.6e12 B/s).  These
 * probes measure what the running GPU delivers, so that the published
 * figures can be checked on the box.
 *
 * Both calls are synchronous: they allocate a small output buffer, launch
 * their kernel twice on the default stream (the second launch is timed with
 * HIP events), free the buffer and return 0, or -1 on a bad argument or a
 * HIP error.
 */
#ifndef SCHEDPROBE_H
#define SCHEDPROBE_H

#ifdef __cplusplus
extern "C" {
#endif

/* 8 blocks of 256 threads per CU; each lane runs `iters` x 128 independent
 * v_add_u32.  Writes lane-operations per second. */
int sched_probe_valu(int iters, double* lane_ops_per_s);

/* 2 blocks of 256 threads per CU (64 KiB of LDS each); each lane reads
 * `iters` x 8 x 16 bytes of LDS, conflict-free.  Writes bytes per second. */
int sched_probe_lds(int iters, double* bytes_per_s);

#ifdef __cplusplus
}
#endif
#endif /* SCHEDPROBE_H */
