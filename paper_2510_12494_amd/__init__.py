"""MI355X (gfx950) two-party publisher/subscriber split-learning step.

``vfl`` is the ctypes binding of the C ABI (include/vfl.h) with the same
names; ``session`` holds the device-side harness (workspace, streams,
resident data).  Both load ``libvfl.so`` built in-tree by ``build.py`` and
fail loudly when it is missing.
"""
