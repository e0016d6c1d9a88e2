/* A plain C99 client of the HIP library: compiled with gcc against the
 * public header and linked against libsdp4.so.  It exercises only argument
 * checks and pure helpers, which never touch a device, and prints one
 * status per line for the test to compare. */
#include <stdint.h>
#include <stdio.h>

#include "sdp4.h"

int main(void)
{
    float *x = (float *)(uintptr_t)0x7f0000000000ull;
    void *codes = (void *)(uintptr_t)0x7f0100000000ull;
    float *scale = (float *)(uintptr_t)0x7f0200000000ull;
    const void *peers[2] = {codes, (const char *)codes + (1 << 20)};
    const float *scales[2] = {scale, scale + (1 << 18)};
    printf("%d\n", sdp4_grad_quant(x, 4096, 3, 256, 128, codes, scale, NULL));           /* EINVAL */
    printf("%d\n", sdp4_grad_quant(x, 4000, 8, 256, 128, codes, scale, NULL));           /* EALIGN */
    printf("%d\n", sdp4_grad_quant(x, 0, 8, 256, 128, codes, scale, NULL));              /* OK */
    printf("%d\n", sdp4_dequant_reduce(17, peers, scales, 4096, 8, 128, 4, 0, 1.0f, codes, scale, NULL,
                                       NULL));                                         /* ERANGE */
    printf("%d\n", sdp4_qwd_encode(x, x, SDP4_BF16 + 1, 4096, 128, codes, scale, scale, NULL)); /* EINVAL */
    printf("%d\n", sdp4_grad_quant_sr(x, 4096, 8, 256, 128, 1, 4, codes, scale, NULL));  /* EALIGN */
    printf("%lld\n", (long long)sdp4_codes_bytes(4096, 4));
    printf("%lld\n", (long long)sdp4_num_groups(4096, 128));
    printf("%s\n", sdp4_status_string(SDP4_ERANGE));
    printf("%d\n", sdp4_last_hip_error());
    return 0;
}
