"""MI355X (gfx950) K-seed DiT denoise-step library.

    paper_2606_19004_amd.ditstep   ctypes binding of libditstep.so (include/ditstep.h)
    paper_2606_19004_amd.build     hipcc build of libditstep.so
"""
