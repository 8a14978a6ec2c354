/*
 * taliesin_debug.h -- exported only by the sabotage build of the library
 * (libtaliesin_sabotage.so, compiled with -DTL_SABOTAGE); the release
 * libtaliesin.so has no such entry point.
 *
 * Sabotage testing (paper, Sec. 3): each defence is attacked with the defence
 * on (the attack must fail), switched off (the attack must succeed) and
 * restored (it must fail again). A defence counts only if all three hold.
 * The sabotage library (built with TL_SABOTAGE) lets a test switch individual load checks off.
 */
#ifndef TALIESIN_DEBUG_H
#define TALIESIN_DEBUG_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TL_CHECK_ROOT 0x01u     /* metadata checksum */
#define TL_CHECK_HEADER 0x02u   /* format, geometry, namespace (tenant + model) */
#define TL_CHECK_POSITION 0x04u /* stored block index */
#define TL_CHECK_KEY 0x08u      /* stored key (the confirmation hash) */
#define TL_CHECK_TOKENS 0x10u   /* byte comparison of the token ids */
#define TL_CHECK_SEGMENT 0x20u  /* payload chunk digests */

/* Switch off the checks in `mask` for every later tl_load of this process
 * (0 restores all of them); returns the previous mask. Length and pointer
 * checks stay on: they guard memory safety, not the content. */
uint32_t tl_debug_disable_checks(uint32_t mask);

#ifdef __cplusplus
}
#endif
#endif /* TALIESIN_DEBUG_H */
