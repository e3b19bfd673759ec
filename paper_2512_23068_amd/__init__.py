"""MI355X-native primal + tangent (forward-mode JVP) scan of a selective
diagonal SSM (Phase Gradient Flow evaluated by Tiled Operator-Space
Evolution).  The compute path is the HIP library ``libpgf.so``; this package
only marshals arguments to it (see ``binding``)."""
