/*
 * kap_diag.h -- measurement helpers of libkap (not part of the method).
 *
 * kap_stream_read -- read `bytes` bytes of device memory at `src` once with
 * 16-byte non-temporal vector loads and fold them into *sink (XOR of all
 * 32-bit words read, XOR-accumulated into the existing value). A plain
 * streaming read of this kind is the practical HBM read ceiling that the
 * attention kernels' bandwidth is compared with.
 *   src: device memory, 16-byte aligned; bytes: a multiple of 16 (0 is a
 *   successful no-op); sink: one device uint32 owned by the caller.
 * Errors (returned before anything is enqueued): KAP_ERR_INVALID_ARGUMENT
 * for a NULL pointer, a misaligned src or a size that is not a multiple of
 * 16; KAP_ERR_HIP if the launch fails. Work is enqueued on `stream`
 * (hipStream_t as void*, NULL = the default stream).
 */
#ifndef KAP_DIAG_H_
#define KAP_DIAG_H_

#include "kap.h"

#ifdef __cplusplus
extern "C" {
#endif

kap_status kap_stream_read(const void *src, size_t bytes, uint32_t *sink, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* KAP_DIAG_H_ */
