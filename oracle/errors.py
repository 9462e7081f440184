"""Error conditions the oracle raises; each corresponds to one status code of the C ABI."""


class OracleError(Exception):
    code = 0


class TagError(OracleError):
    """Malformed slot tags: unit id outside [-1, U), modality above 4, or a live unit whose
    slots are not one contiguous run in temporal (slot) order."""
    code = -17


class BudgetError(OracleError):
    """The protected (system) units alone exceed the retention budget."""
    code = -16


class CapacityError(OracleError):
    """Retained history plus the new chunk does not fit the destination pool."""
    code = -5
