/*
 * f2probe.h -- C ABI of the ceiling probes used beside the vendor peaks when a
 * measured rate is turned into a roofline fraction.  They compute nothing of
 * the method: one kernel streams a buffer through HBM (the achievable memory
 * bandwidth), one issues a long run of independent 32-bit bitwise VALU
 * operations (the achievable integer issue rate that the blocked elimination
 * of wide contexts is measured against), and one reads or writes at random
 * positions of a buffer (the achievable rate of scattered accesses, which bounds
 * the context-grouped encode).
 *
 * Conventions: pointers are DEVICE memory owned by the caller, work is
 * enqueued on `stream` (a hipStream_t passed as void*, NULL = null stream),
 * a negative return means nothing was enqueued.
 */
#ifndef F2PROBE_H
#define F2PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * dst[i] = src[i] for i < words (uint64 words), 16 bytes per lane per access,
 * coalesced, a grid-stride loop over the buffer.  Both buffers 16-byte aligned
 * and not overlapping.  Returns 0, -1 (bad argument) or -3 (HIP error).
 */
int f2probe_copy(const uint64_t* src, uint64_t* dst, int64_t words, void* stream);

/*
 * Integer issue rate.  `blocks` workgroups of 256 threads; every thread runs
 * `iters` iterations of 16 dependent-free 32-bit bitwise instructions of the
 * kind `op` selects (0: two-input XOR, v_xor_b32; 1: three-input bitwise
 * function, v_bitop3_b32 computing a ^ b ^ c) over 16 values, then stores one
 * word to out[global thread index] so that nothing is optimised away.
 * Instructions issued = blocks * 256 * iters * 16.
 * out holds blocks * 256 uint32 words.  Returns 0, -1 or -3.
 */
int f2probe_bitops(uint32_t* out, int32_t blocks, int32_t iters, int32_t op, void* stream);

/*
 * Scattered accesses.  `blocks` workgroups of 256 threads; thread t makes `per`
 * accesses at slots given by a hash of (t, access index) modulo the number of
 * slots in the first `bytes` bytes of buf: op 0 reads 32 bytes at a 32-byte slot
 * (all of them XOR-folded into out[t], so out holds blocks * 256 uint64 words),
 * op 1 writes 16 bytes at a 16-byte slot (out unused, may be NULL).  Accesses =
 * blocks * 256 * per.  buf 16-byte aligned, bytes >= 32.  Returns 0, -1 or -3.
 */
int f2probe_scatter(uint64_t* buf, int64_t bytes, int32_t blocks, int32_t per, int32_t op, uint64_t* out,
                    void* stream);

#ifdef __cplusplus
}
#endif
#endif /* F2PROBE_H */
