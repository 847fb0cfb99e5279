/*
 * stage_alloc.h -- the fine-grained allocation scheduler of arXiv 2512.21835 (Section III-D,
 * Alg. 1, with the cost model of Eq. (1) and the overlap window of Eq. (2)) as a host function
 * of the stage library.
 *
 * Given the decoder layers of a model and a chain of devices, each with its memory, its time to
 * compute one layer and its time to load one offloaded layer block, the scheduler decides how
 * many layers every device runs, how many of them it offloads (reloading them every decoding
 * step while its other work runs), whether an offloaded layer is offloaded whole or only its MHA
 * or MLP block, and the number of interleaved stages per device (#Stage):
 *   1. every device first takes the layers its memory holds;
 *   2. for each #Stage s, a dynamic program spreads the remaining layers over the devices as
 *      offloaded layers, minimising the loading delay the overlap windows (Eq. (2)) leave
 *      uncovered (Eqs. (3)-(4));
 *   3. while the device with the longest loading time has memory left, one of its offloaded
 *      layers keeps a block resident (block-level offloading);
 *   4. the s of least T_total (Eq. (1)) wins.
 * Times are integers in any one unit (e.g. ns); memory in bytes.  The readings taken where the
 * printed algorithm is ambiguous are stated at stage_allocate.
 *
 * Conventions as in stage.h: 0 (STAGE_OK) or a negative stage_status; nothing throws.  This
 * function only computes: no GPU, no allocation visible to the caller, no state.
 */
#ifndef PAPER_2512_21835_STAGE_ALLOC_H
#define PAPER_2512_21835_STAGE_ALLOC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int64_t mem_bytes;    /* Mem_i: memory for weights on the device */
    int64_t comp_layer;   /* comp of one decoder layer on the device, per decoding step, >= 0 */
    int64_t load_mha;     /* load of one MHA block onto the device (p_A of a layer), > 0 */
    int64_t load_mlp;     /* load of one MLP block (p_M of a layer), > 0 */
} stage_alloc_device;

typedef struct {
    int32_t n_layers;     /* |L|, >= 1 */
    int64_t mha_bytes;    /* p_A * l_size, > 0 */
    int64_t mlp_bytes;    /* p_M * l_size, > 0; l_size = mha_bytes + mlp_bytes */
    int64_t comm;         /* h_size / bw_net: passing one layer output between devices, >= 0 */
    int32_t n_devices;    /* |D|, 1 ..  STAGE_ALLOC_MAX_DEVICES */
    const stage_alloc_device *devices;  /* in pipeline order */
} stage_alloc_input;

#define STAGE_ALLOC_MAX_DEVICES 64
#define STAGE_ALLOC_MAX_LAYERS 4096

typedef struct {
    int32_t first_layer;  /* the device runs layers [first_layer, first_layer + assigned) */
    int32_t assigned;     /* |L_i|: retained plus offloaded layers */
    int32_t offloaded;    /* |L~_i|: layers (or blocks of them) reloaded every decoding step */
    int32_t mha_only;     /* of the offloaded layers, those whose MLP block stays resident */
    int32_t mlp_only;     /* of the offloaded layers, those whose MHA block stays resident */
} stage_alloc_plan;

/* Runs Alg. 1.  Writes one plan per device into out[n_devices], the chosen #Stage into *n_stage
   and T_total of Eq. (1) under that plan into *t_total.
   Readings (the printed algorithm leaves these open or is inconsistent):
   - capacity C_i = floor(Mem_i / l_size) layers; the layers beyond sum(C_i), L_Left, are what the
     dynamic program spreads; if there are none, devices take layers in order up to capacity,
     nothing is offloaded and #Stage = 1;
   - #Stage ranges over 2 .. min(max(2, |L_Left|), ceil(|L| / |D|));
   - the overlap windows (Eq. (2)) are taken before offloading: T_i^idle = C_i*comp_i +
     sum over the other devices of C_i'*comp_i' + |D|*comm;
   - the dynamic program clamps at zero from the first device on (Eq. (3) as a clamped
     transition from F(0) = 0, like the later transitions); ties keep the larger share for the
     later device (the printed "<=" update over increasing k);
   - a #Stage is infeasible when a device's layers per stage exceed its capacity:
     C_i + |L~_i| > s * C_i (the printed test, with its comparison read as the failure case);
   - refinement: device loading time T_i = whole*(load_mha + load_mlp) + mha_only*load_mha +
     mlp_only*load_mlp; the device with the largest T_i (lowest index on ties) converts one
     whole offloaded layer: to MHA-only offloading if its leftover memory Mem_i - C_i*l_size
     holds an MLP block (T_i drops by load_mlp), else to MLP-only offloading if it holds an MHA
     block (T_i drops by load_mha), else the refinement ends (also when that device has no whole
     offloaded layer left); the saving is the block that stops being loaded;
   - T_total = sum_i comp_i*|L_i| + s*|D|*comm + max_i max(0, T_i - (comp_i*C_i + sum over the
     other devices of comp_i'*|L_i'| + |D|*comm)); the least T_total wins, ties to the smaller s.
   EINVAL: bad input; ERANGE: no #Stage is feasible (or |L| exceeds what the range allows).
   Integer arithmetic throughout (EINVAL if it would overflow int64). */
int stage_allocate(const stage_alloc_input *in, stage_alloc_plan *out, int32_t *n_stage, int64_t *t_total);

#ifdef __cplusplus
}
#endif

#endif /* PAPER_2512_21835_STAGE_ALLOC_H */
