/* Seeded synthetic routing-id generator (host twin).
 *
 * Input generation only: this file holds none of the planner's arithmetic.
 * The device twin (gen_ids_dev.hip) implements the same definition and must
 * produce bit-identical ids; a test compares the two.
 *
 * Definition.  For problem b with seed `seed`, source rank r, token t and
 * draw d (0 <= d < k), attempt a = 0, 1, ... draws
 *     u = upper 32 bits of splitmix64_at(seed, ((r*T + t)*k + d) * 2^20 + a)
 * and maps u to the smallest expert e with u < thr[e] (thr is a
 * non-decreasing uint64 table with thr[E-1] = 2^32).  A draw equal to an
 * expert already chosen for this token is redrawn with a + 1, so each token
 * gets k distinct experts (successive sampling without replacement in
 * proportion to the table's weights).  After 2^20 - 1 rejected attempts the
 * smallest unused expert id is taken (never reached for the shipped tables).
 *
 * splitmix64_at(seed, i) is the i-th output (0-based) of SplitMix64
 * (Steele, Lea, Flood, OOPSLA 2014) started from state `seed`:
 *     z = seed + (i + 1) * 0x9E3779B97F4A7C15
 *     z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9
 *     z = (z ^ (z >> 27)) * 0x94D049BB133111EB
 *     return z ^ (z >> 31)
 * Ids are written as int32 out[(r - r0)][t][d] for r in [r0, r1).
 */
#ifndef TAOT_WORKLOADS_GEN_IDS_H
#define TAOT_WORKLOADS_GEN_IDS_H
#include <stdint.h>

#define GEN_MAX_K 32
#define GEN_ATTEMPT_BITS 20

#ifdef __cplusplus
extern "C" {
#endif

uint64_t gen_splitmix64_at(uint64_t seed, uint64_t i);

/* Returns 0 on success, -1 on invalid arguments (k > GEN_MAX_K, k > E, ...). */
int gen_ids_host(const uint64_t* thr, int32_t E, uint64_t seed, int32_t R, int64_t T,
                 int32_t k, int32_t r0, int32_t r1, int32_t* out);

#ifdef __cplusplus
}
#endif
#endif
