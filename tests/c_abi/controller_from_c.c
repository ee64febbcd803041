/* Drives the interval controller through the C ABI with raw structs: reads one
 * autoloco_controller_cfg and then autoloco_observation records from stdin,
 * writes every autoloco_decision to stdout.  Every seventh observation the
 * controller state is saved, the controller destroyed and a fresh one (created
 * with the default configuration) loaded from the checkpoint, so the
 * checkpoint path runs under the same checks as the decisions.  Host code only:
 * it links the controller and scalar sources, no device library.
 * Exit status: 0 on success, 2..9 for the step that failed. */
#include <stdio.h>
#include <stdlib.h>

#include "autoloco.h"

static autoloco_controller* reload(autoloco_controller* c) {
    size_t len = 0;
    if (autoloco_controller_save(c, NULL, &len) != AUTOLOCO_OK || len == 0) return NULL;
    void* buf = malloc(len);
    if (buf == NULL) return NULL;
    autoloco_controller* fresh = NULL;
    autoloco_controller_cfg def;
    autoloco_controller_default_cfg(&def);
    int ok = autoloco_controller_save(c, buf, &len) == AUTOLOCO_OK &&
             autoloco_controller_create(&def, &fresh) == AUTOLOCO_OK &&
             autoloco_controller_load(fresh, buf, len) == AUTOLOCO_OK;
    free(buf);
    autoloco_controller_destroy(c);
    if (!ok) {
        autoloco_controller_destroy(fresh);
        return NULL;
    }
    return fresh;
}

int main(void) {
    autoloco_controller_cfg cfg;
    if (fread(&cfg, sizeof cfg, 1, stdin) != 1) return 2;
    autoloco_controller* c = NULL;
    if (autoloco_controller_create(&cfg, &c) != AUTOLOCO_OK) return 3;
    autoloco_decision d;
    if (autoloco_select_interval(c, NULL, &d) != AUTOLOCO_OK) return 4;
    if (fwrite(&d, sizeof d, 1, stdout) != 1) return 5;
    autoloco_observation o;
    long i = 0;
    while (fread(&o, sizeof o, 1, stdin) == 1) {
        if (++i % 7 == 0 && (c = reload(c)) == NULL) return 6;
        if (autoloco_select_interval(c, &o, &d) != AUTOLOCO_OK) return 7;
        if (fwrite(&d, sizeof d, 1, stdout) != 1) return 8;
    }
    autoloco_controller_destroy(c);
    return ferror(stdin) ? 9 : 0;
}
