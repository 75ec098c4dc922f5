// mq_probe_read: a plain streaming read of device memory, for measuring the
// floor under the decode kernel (the time a grid of that shape needs just to
// bring the same number of bytes in from HBM).  Not a step of the method.
//
// Block b reads bytes [b*per, (b+1)*per) of the buffer, per = bytes/blocks
// rounded up to 1 KiB.  Its waves take 1 KiB wave loads in turn (lane i
// reads 16 bytes at 16*i), `unroll` loads per lane in flight per round, all
// through a buffer descriptor over the whole buffer, so loads past its end
// return zeros.  The loads carry the non-temporal cache policy, as the
// decode kernels' weight loads do.  Each wave writes the XOR of what it read to one word of
// `sink`, so no load can be dropped.
#include "mq_internal.h"

namespace mq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

template <int U>
__global__ void probe_read_kernel(const int8_t* src, int64_t bytes, int64_t per, int32_t* sink)
{
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int waves = blockDim.x >> 6;
    const int64_t b0 = (int64_t)blockIdx.x * per;
    const int64_t len = bytes - b0 < per ? bytes - b0 : per;
    // descriptor over this block's range: loads past it return zeros
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(src + b0), (short)0, (int)(len > 0 ? len : 0), 0x00020000);
    v4i x = {0, 0, 0, 0};
    const int64_t round = (int64_t)U * waves * 1024;
    for (int64_t base = 0; base < len; base += round) {
        v4i v[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            v[u] = __builtin_amdgcn_raw_buffer_load_b128(
                r, (uint32_t)(base + ((int64_t)u * waves + wave) * 1024 + lane * 16), 0, 2);
#pragma unroll
        for (int u = 0; u < U; ++u) x ^= v[u];
    }
    int s = x[0] ^ x[1] ^ x[2] ^ x[3];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) s ^= __shfl_xor(s, o);
    if (lane == 0) sink[(int64_t)blockIdx.x * waves + wave] = s;
}

}  // namespace
}  // namespace mq

extern "C" mq_status mq_probe_read(const void* src, int64_t bytes, int32_t blocks, int32_t waves,
                                   int32_t unroll, int32_t* sink, void* stream)
{
    if (bytes < 0 || blocks <= 0 || waves <= 0 || waves > 16) return MQ_ERR_INVALID_ARG;
    if (unroll != 1 && unroll != 2 && unroll != 4 && unroll != 8 && unroll != 16)
        return MQ_ERR_INVALID_ARG;
    if (!sink || (bytes > 0 && !src)) return MQ_ERR_INVALID_ARG;
    const int64_t per = ((bytes + blocks - 1) / blocks + 1023) / 1024 * 1024;
    if (per >= ((int64_t)1 << 31)) return MQ_ERR_UNSUPPORTED;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int8_t* p = static_cast<const int8_t*>(src);
    const dim3 g((unsigned)blocks), t((unsigned)(64 * waves));
    switch (unroll) {
    case 1: mq::probe_read_kernel<1><<<g, t, 0, s>>>(p, bytes, per, sink); break;
    case 2: mq::probe_read_kernel<2><<<g, t, 0, s>>>(p, bytes, per, sink); break;
    case 4: mq::probe_read_kernel<4><<<g, t, 0, s>>>(p, bytes, per, sink); break;
    case 8: mq::probe_read_kernel<8><<<g, t, 0, s>>>(p, bytes, per, sink); break;
    default: mq::probe_read_kernel<16><<<g, t, 0, s>>>(p, bytes, per, sink); break;
    }
    return hipGetLastError() == hipSuccess ? MQ_OK : MQ_ERR_HIP;
}
