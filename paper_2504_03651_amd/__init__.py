"""MI355X (gfx950) mixed paged-attention iteration of the Echo serving system.

Modules: ``workload`` (seeded synthetic inputs), ``echo`` (ctypes binding of
libecho.so), ``session`` (device state of one iteration), ``build`` (hipcc
build of the library).  Importing the package loads nothing; the first call
into ``echo`` loads the library and fails loudly if it is missing.
"""
