/*
 * CPU oracle for the retrieval-drafted verify step. TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, fp64 reference of what the decoding hot path computes. Only
 * the test suite, the smoke check and the benchmark's CPU-baseline leg use
 * it. It shares no code, header or table with the HIP library.
 */
#ifndef PF_ORACLE_H
#define PF_ORACLE_H
#include <stdint.h>

typedef struct or_model {
  int L, H, nq, nkv, hd, F, V;
  double theta, eps;
  int bf16; /* 1: weights and cache are bf16 bit patterns and activations are
               rounded to bf16 at the contract points; 0: everything fp32 */
  const void *embed;   /* [V][H] */
  const void *lm_head; /* [V][H] */
  const void *wqkv;    /* [L][nq*hd + 2*nkv*hd][H] */
  const void *wo;      /* [L][H][nq*hd] */
  const void *wgu;     /* [L][2F][H]: gate rows, then up rows */
  const void *wd;      /* [L][H][F] */
  const float *attn_norm, *ffn_norm; /* [L][H] */
  const float *final_norm;           /* [H] */
} or_model;

#endif
