/*
 * ra_oracle_fs.h -- the oracle's Fiat-Shamir transcript (ra_oracle_fs.c).
 * TEST INFRASTRUCTURE ONLY; shared by the oracle's own files, never by the
 * product library.
 */
#ifndef RA_ORACLE_FS_H
#define RA_ORACLE_FS_H
#include <stddef.h>
#include <stdint.h>

/* S: the 32-byte state; Q: the bytes absorbed since the last draw. */
typedef struct {
    uint8_t S[32];
    uint32_t qlen;
    uint8_t Q[1024];
} orc_fs;

void orc_sha256(const uint8_t *msg, size_t len, uint8_t out[32]);
void orc_fs_init(orc_fs *t, const uint8_t domain[32]);
int orc_fs_absorb(orc_fs *t, const uint8_t *m, uint32_t len);
void orc_fs_draw(orc_fs *t, uint64_t out[2]);
int orc_witness_root(const int64_t *R, const int64_t *Rm, const int64_t *Y, const int64_t *Z, const uint64_t *words,
                     int64_t N, uint8_t out[32]);

#endif
