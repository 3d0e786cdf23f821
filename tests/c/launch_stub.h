/* Controls of the CPU stand-in for the GPU launches (launch_stub.cpp). */
#ifndef KAMERA_LAUNCH_STUB_H
#define KAMERA_LAUNCH_STUB_H
#ifdef __cplusplus
extern "C" {
#endif
void stub_set_launch_error(int hip_error);   /* 0: launches succeed */
long stub_launches(void);                    /* launches so far, all threads */
int stub_last_rehydrate_row_group(void);     /* this thread's last rehydrate */
long long stub_last_rehydrate_tasks(void);
int stub_last_rehydrate_block_tiles(void);   /* 0: persistent schedule */
#ifdef __cplusplus
}
#endif
#endif
