/*
 * tp_probe.h -- hardware probes behind the roofline ceilings quoted for the
 * kernels (measurement tooling; libtpprobe.so, separate from libtp.so).
 * Device pointers, asynchronous on `stream` (a hipStream_t); 0 = launched,
 * -1 = bad arguments, -4 = launch error.  The caller times the launches.
 */
#pragma once
#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* `blocks` workgroups of four waves, each issuing iters x 8 independent
 * v_mfma_f32_16x16x32_bf16 on register operands.  out: blocks * 256 floats
 * (written only under a condition the data never meets). */
int tpp_mfma_issue(int blocks, int iters, float *out, void *stream);

/* Algorithmic FLOPs of one tpp_mfma_issue launch. */
double tpp_mfma_issue_flops(int blocks, int iters);

/* The same with v_mfma_f32_32x32x16_bf16, four independent accumulators. */
int tpp_mfma32_issue(int blocks, int iters, float *out, void *stream);
double tpp_mfma32_issue_flops(int blocks, int iters);

/* Issue-rate sweep: `blocks` workgroups of `waves` waves (1..16), each wave
 * issuing iters x nacc back-to-back MFMAs of shape m (16:
 * v_mfma_f32_16x16x32_bf16, 32: v_mfma_f32_32x32x16_bf16) into nacc
 * (1, 2, 4 or 8) independent accumulators, with one A/B operand pair per
 * accumulator (distinct != 0) or one pair shared by all.  out:
 * blocks * waves * 64 floats (written only under a condition the data never
 * meets); clk[0..1] (device): the shader-clock and the 100 MHz-clock ticks
 * wave 0 of workgroup 0 spent in its loop. */
int tpp_mfma_sweep(int m, int nacc, int distinct, int blocks, int waves, int iters, float *out,
                   unsigned long long *clk, void *stream);
double tpp_mfma_sweep_flops(int m, int nacc, int blocks, int waves, int iters);

/* `blocks` workgroups of eight waves; wave w streams 1-KiB fragments
 * f = 0 .. frags_per_wave-1 of buf + w * frags_per_wave KiB, reps times,
 * 16 loads in flight.  buf >= 8 * frags_per_wave KiB (every workgroup reads
 * the same bytes, so they come from L2 after the first pass); out:
 * blocks * 512 * 16 bytes.  Bytes pulled per workgroup:
 * 8 * frags_per_wave * 1024 * reps. */
int tpp_l2_stream(const void *buf, size_t buf_bytes, int frags_per_wave, int reps, int blocks,
                  void *out, void *stream);

/* Workgroup handoff latency: 2 * pairs workgroups of one wave; b and
 * b ^ stride (stride a power of two, 2 * stride dividing 2 * pairs) pass a
 * counter back and forth `rounds` times through one flag word (flags:
 * pairs * 32 ints, zeroed by the caller) with agent-scope release/acquire
 * (mode 0) or relaxed agent-scope atomics (mode 1).  Every wait gives up
 * after spin_limit polls.  out: 2 * pairs records {uint32 xcc, uint32
 * timeouts, uint64 ticks of the 100 MHz clock over the loop}. */
int tpp_pingpong(int mode, int pairs, int stride, int rounds, int spin_limit, int *flags,
                 void *out, void *stream);

/* The handoff with a 16 KiB payload per turn (1024 16-byte words written by
 * one side, read and checked by the other): payload accesses plain stores
 * and L1-bypassing loads (mode 0) or device-scope stores and loads (mode 1);
 * the flag as mode 1 of tpp_pingpong.  flags: pairs * 32 ints (zeroed);
 * data: pairs * 2 * 1024 16-byte words; out: 2 * pairs records {uint32 xcc,
 * uint32 timeouts, uint64 ticks, uint32 stale words read, uint32 pad}. */
int tpp_pingpong_data(int mode, int pairs, int stride, int rounds, int spin_limit, int *flags,
                      void *data, void *out, void *stream);

/* tpp_l2_stream with an agent-scope acquire (mode 1) or release (mode 2)
 * fence every `every` fragments of each wave (mode 0: none). */
int tpp_l2_stream_fence(const void *buf, size_t buf_bytes, int frags_per_wave, int reps,
                        int blocks, int mode, int every, void *out, void *stream);

/* A plain copy of `bytes` (a multiple of 16; both pointers 16-byte
 * aligned) from src to dst by `blocks` workgroups of 256 threads, 16 bytes
 * per lane per access, four loads in flight, non-temporal. */
int tpp_copy(const void *src, void *dst, size_t bytes, int blocks, void *stream);

#ifdef __cplusplus
}
#endif
