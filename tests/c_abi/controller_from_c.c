/* Drives the interval controller through the C ABI with raw structs: reads one
 * autoloco_controller_cfg and then autoloco_observation records from stdin,
 * writes every autoloco_decision to stdout.  Every seventh observation the
 * controller state is saved, the controller destroyed and a fresh one (created
 * with the default configuration) loaded from the checkpoint, so the
 * checkpoint path runs under the same checks as the decisions.  Host code only:
 * it links the controller and scalar sources, no device library.
 * Exit status: 0 on success, 2..9 for the step that failed.
 *
 * With the argument "load": reads a checkpoint from stdin, loads it into a
 * controller created with the default configuration and writes the status
 * (int32); when the load succeeds it takes one more decision on a fixed
 * observation and writes it too, so a loaded state runs under the same
 * checks. */
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

static int load_mode(void) {
    static unsigned char blob[1 << 16];
    const size_t len = fread(blob, 1, sizeof blob, stdin);
    autoloco_controller_cfg def;
    autoloco_controller_default_cfg(&def);
    autoloco_controller* c = NULL;
    if (autoloco_controller_create(&def, &c) != AUTOLOCO_OK) return 3;
    const int32_t st = autoloco_controller_load(c, blob, len);
    if (fwrite(&st, sizeof st, 1, stdout) != 1) return 5;
    if (st == AUTOLOCO_OK) {
        const autoloco_observation o = {1e-2, 4.0, 1.0, 524288000.0, 500, 1};
        autoloco_decision d;
        const int32_t s2 = autoloco_select_interval(c, &o, &d);
        if (fwrite(&s2, sizeof s2, 1, stdout) != 1) return 5;
        if (s2 == AUTOLOCO_OK && fwrite(&d, sizeof d, 1, stdout) != 1) return 8;
    }
    autoloco_controller_destroy(c);
    return 0;
}

int main(int argc, char** argv) {
    if (argc > 1 && argv[1][0] == 'l') return load_mode();
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
