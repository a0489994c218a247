"""MI355X-native pipeline-stage forward pass (hand-written HIP for gfx950).

Importing the package loads nothing native; ``paper_2606_18600_amd.stage``
loads the HIP library and fails loudly if it is missing.
"""
