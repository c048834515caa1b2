"""ID Balancing router step and bias controller for AMD MI355X (gfx950).

* ``binding`` -- ctypes binding of the C ABI in ``include/idb.h`` (libidb.so)
* ``pipeline`` -- device buffers and the calls of one router + controller step
* ``synth`` -- seeded synthetic inputs (no method arithmetic)
* ``build`` -- compiles libidb.so for gfx950
"""
